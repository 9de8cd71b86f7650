"""SJF's dispatch-tick loop over the whole drift workload on the GPU.

4,194,304 requests arriving at 5,000/s, 4,096 groups, 10 ms ticks of 32: the
pending set peaks near 1.3 M requests and the loop runs 131,088 ticks, more
than the oracle can replay tick by tick (it re-sorts the pending set every
tick). What holds at any size is checked instead, with the oracle's own
score, calibrate and order functions on the GPU's output:

* every request is dispatched once, at a tick at or after its arrival, and
  each tick dispatches min(32, pending) requests;
* the final factors equal the oracle's Eq. (5) with the ratio of Eq. (6)
  applied to the completions in the GPU's dispatch order (bit-exact);
* at sampled ticks (the first, the busiest, the last and random ones) the
  batch is exactly the first min(32, pending) of the oracle's SJF order of
  that tick's pending set, with budgets of Eq. (1)-(2) scored from the
  factors as they stood at that tick (the same calibration's trace).
"""
import numpy as np
import pytest

import workloads as synth
from tests import wl
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu

SJF = 3


def test_sjf_drift_workload_full(oracle):
    from paper_2606_02982_amd import driftsched as ds
    b = wl.load("drift4m", with_text=False)
    n, G, batch, alpha = b.n, b.n_groups, 32, b.alphas[0]
    ticks = synth.sim_ticks(b.arrival)
    print("simulate SJF n=%d ticks=%d batch=%d" % (n, len(ticks), batch), flush=True)
    p = ds.sim_params(SJF, batch=batch, alpha=alpha, f_ref=b.f_ref)
    st = dev(np.ones(G))
    seq, tick_of, nd = ds.simulate(dev(b.arrival), dev(b.tier), dev(b.words), dev(b.category),
                                   dev(b.tenant), dev(b.group), dev(b.observed), dev(b.t_base),
                                   dev(b.s_tenant), st, dev(ticks), p)
    nd = int(host(nd)[0])
    seq = host(seq, np.uint32)[:nd].astype(np.int64)
    tick_of = host(tick_of)
    state = host(st)
    print("dispatched %d; checking" % nd, flush=True)

    # every request once, after its arrival, min(batch, pending) per tick
    assert nd == n
    assert np.array_equal(np.sort(seq), np.arange(n))
    tk = tick_of[seq]
    assert tk.min() >= 0 and np.all(np.diff(tk) >= 0)
    assert np.all(b.arrival[seq] <= ticks[tk])
    per_tick = np.bincount(tk, minlength=len(ticks))
    arrived = np.searchsorted(np.sort(b.arrival), ticks, side="right")
    before = np.concatenate([[0], np.cumsum(per_tick)[:-1]])
    assert np.array_equal(per_tick, np.minimum(batch, arrived - before))

    # the factors: the oracle's calibration over the dispatch sequence
    est_base = wl.est_base(b)
    ev_g = b.group[seq]
    w_state, trace = oracle.calibrate(ev_g, est_base[seq], b.observed[seq], alpha, np.ones(G))
    assert np.array_equal(state, w_state)

    # sampled ticks against the oracle's SJF order of the pending set
    rng = np.random.default_rng(0)
    busiest = int(np.argmax(arrived - before))
    sample = np.unique(np.concatenate([[0, 1, busiest, len(ticks) - 200],
                                       rng.choice(len(ticks) - 16, 20, replace=False)]))
    last = np.full(G, -1, np.int64)      # each group's last event before the tick
    done = 0
    for k in sample:
        D, m = int(before[k]), int(per_tick[k])
        np.maximum.at(last, ev_g[done:D], np.arange(done, D))
        done = D
        if m == 0:
            continue
        st_k = np.where(last >= 0, trace[np.maximum(last, 0)], 1.0)
        pend = np.flatnonzero((b.arrival <= ticks[k]) & (tick_of >= k))
        bud = oracle.score(b.words[pend], b.category[pend], b.tenant[pend], b.group[pend], b.t_base,
                           b.s_tenant, st_k, f_ref=b.f_ref)[2]
        # the order's first m are among the requests with the m smallest budgets
        cand = np.flatnonzero(bud <= np.partition(bud, m - 1)[m - 1])
        perm, _ = oracle.order(SJF, b.tier[pend[cand]], b.arrival[pend[cand]], bud[cand])
        want = pend[cand[perm[:m]]]
        assert np.array_equal(seq[D:D + m], want), "tick %d (pending %d)" % (k, len(pend))
        print("tick %d: pending %d, batch %d ok" % (k, len(pend), m), flush=True)
