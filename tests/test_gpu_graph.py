"""The whole admission step captured in a HIP graph and replayed.

Every launch of the library goes on the caller's stream and none is a
memset, so a step can be captured once and replayed. Each replay must give
the eager step's results exactly: replays are interleaved with eager work
and synchronisations, and every replay is checked.
"""
import numpy as np
import pytest
import torch

from tests import wl
from tests.gpu_util import dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


@pytest.mark.parametrize("schedule", ["serial", "overlap"])
def test_step_graph_replays_equal_eager(ds, schedule):
    b = wl.load("batch4k")
    N = b.n
    text, offsets = dev(b.text), dev(b.offsets)
    ev_group, ev_est, ev_obs = dev(b.ev_group), dev(b.ev_est), dev(b.ev_obs)
    category, tenant, group = dev(b.category), dev(b.tenant), dev(b.group)
    t_base, s_tenant = dev(b.t_base), dev(b.s_tenant)
    tier, arrival = dev(b.tier), dev(b.arrival)
    params = ds.order_params(weights=tuple(int(w) for w in b.weights),
                             tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate,
                             t_now=b.t_now, aging_floor=b.aging_floor)
    ws = {op: ds.workspace(op, N, b.n_groups) for op in range(5)}

    def buffers():
        return dict(counts=torch.empty(N, dtype=torch.int32, device="cuda"),
                    state=torch.ones(b.n_groups, dtype=torch.float64, device="cuda"),
                    trace=torch.empty(N, dtype=torch.float64, device="cuda"),
                    sc=tuple(torch.empty(N, dtype=torch.float64, device="cuda") for _ in range(3)) +
                    (torch.empty(N, dtype=torch.uint8, device="cuda"),),
                    perms={p: torch.empty(N, dtype=torch.int32, device="cuda") for p in range(5)})

    aux = torch.cuda.Stream()
    ws_aux = ds.workspace(ds.OP_ORDER_MULTI, N, b.n_groups)

    def serial(o):
        o["state"].fill_(1.0)   # a fill kernel, not a memset
        ds.characterize(text, offsets, counts=o["counts"], ws=ws[ds.OP_CHARACTERIZE])
        ds.calibrate(ev_group, ev_est, ev_obs, b.alphas[0], o["state"], trace=o["trace"],
                     ws=ws[ds.OP_CALIBRATE])
        ds.score(o["counts"], category, tenant, group, t_base, s_tenant, o["state"], out=o["sc"])
        ds.order_multi((0, 1, 2, 3, 4), tier, arrival, o["sc"][2], params=params, perms=o["perms"],
                       ws=ws[ds.OP_ORDER_MULTI])

    def overlap(o):
        # calibrate and the budget-free orders on a second stream beside
        # characterize; score and SJF after the join
        o["state"].fill_(1.0)
        main_s = torch.cuda.current_stream()
        aux.wait_stream(main_s)
        with torch.cuda.stream(aux):
            ds.calibrate(ev_group, ev_est, ev_obs, b.alphas[0], o["state"], trace=o["trace"],
                         ws=ws[ds.OP_CALIBRATE])
            ds.order_multi((0, 1, 2, 4), tier, arrival, params=params, perms=o["perms"], ws=ws_aux)
        ds.characterize(text, offsets, counts=o["counts"], ws=ws[ds.OP_CHARACTERIZE])
        main_s.wait_stream(aux)
        ds.score(o["counts"], category, tenant, group, t_base, s_tenant, o["state"], out=o["sc"])
        ds.order_multi((3,), tier, arrival, o["sc"][2], fifo=o["perms"][0], params=params,
                       perms=o["perms"], ws=ws[ds.OP_ORDER_MULTI])

    step = serial if schedule == "serial" else overlap

    def snapshot(o):
        out = [o["counts"], o["state"], o["trace"]] + list(o["sc"]) + [o["perms"][p] for p in range(5)]
        return [t.cpu().clone() for t in out]

    ref = buffers()
    serial(ref)
    torch.cuda.synchronize()
    want = snapshot(ref)

    out = buffers()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(out)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            step(out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    scratch = buffers()
    for rep in range(4):
        for t in [out["counts"], out["trace"]] + list(out["sc"][:3]) + list(out["perms"].values()):
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = snapshot(out)
        for i, (a, w) in enumerate(zip(got, want)):
            assert torch.equal(a, w), "replay %d: output %d differs" % (rep, i)
        step(scratch)   # eager work between the replays
        torch.cuda.synchronize()
    assert np.array_equal(want[0].numpy().view(np.uint32), b.words)


@pytest.mark.parametrize("mode", ["smooth", "stride"])
@pytest.mark.parametrize("n", [65536, 300000])
def test_order_modes_graph_replays(ds, mode, n):
    # the smooth table is built by the last scatter tile to finish (a ticket
    # cleared by the sample launch) or by the plan block: every replay must
    # give the eager orders
    rng = np.random.default_rng(n)
    tier = dev(rng.integers(0, 4, n).astype(np.uint8))
    arrival = dev(np.round(rng.uniform(0, 50, n), 3))
    budget = dev(np.round(rng.uniform(1, 3000, n), 1))
    params = ds.order_params(n_tiers=4, weights=(5, 3, 2, 1), tier_priority=(0.0, 1.0, 2.0, 3.0),
                             aging_rate=0.01, t_now=50.0, weighted_mode=mode)
    ws = ds.workspace(ds.OP_ORDER_MULTI, n, 0)
    print("graph order_multi mode=%s n=%d" % (mode, n), flush=True)
    want, _ = ds.order_multi((0, 1, 2, 3, 4), tier, arrival, budget, params=params, ws=ws)
    torch.cuda.synchronize()
    want = {p: t.cpu().clone() for p, t in want.items()}
    perms = {p: torch.empty(n, dtype=torch.int32, device="cuda") for p in range(5)}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ds.order_multi((0, 1, 2, 3, 4), tier, arrival, budget, params=params, perms=perms, ws=ws)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            ds.order_multi((0, 1, 2, 3, 4), tier, arrival, budget, params=params, perms=perms, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in perms.values():
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for p in range(5):
            assert torch.equal(perms[p].cpu(), want[p]), "replay %d policy %d" % (rep, p)
        ds.order_multi((2,), tier, arrival, budget, params=params, ws=ws)   # eager work between replays
        torch.cuda.synchronize()


def test_simulate_multi_graph_replays(ds):
    """Twelve tick loops in one ds_simulate_multi launch (more runs than one
    kernel argument block holds: their arguments are copied into the
    workspace by small kernels) captured in a graph; every replay, with
    eager calls in between, equals the eager call."""
    from tests.test_gpu_sim import random_inputs
    n, R = 3000, 12
    x = random_inputs(17, n, G=5)
    d = {k: dev(np.asarray(v)) for k, v in x.items() if k != "state"}
    ticks = dev(np.linspace(0.05, 12.0, 120))
    params = [ds.sim_params(r % 5, batch=32 if r % 4 else 8, alpha=0.05 + 0.03 * r, n_tiers=3,
                            weights=(3, 2, 1), tier_priority=(0.0, 1.0, 2.0), aging_rate=0.3)
              for r in range(R)]
    ws = ds.workspace(ds.OP_SIMULATE_MULTI, n, R)
    states = [torch.ones(5, dtype=torch.float64, device="cuda") for _ in range(R)]

    def call():
        for st in states:
            st.fill_(1.0)   # a fill kernel, not a memset
        return ds.simulate_multi(d["arrival"], d["tier"], d["counts"], d["category"], d["tenant"],
                                 d["group"], d["observed"], d["t_base"], d["s_tenant"], states, ticks,
                                 params, ws=ws)

    print("graph simulate_multi: %d runs, n=%d" % (R, n), flush=True)
    outs, nd = call()
    torch.cuda.synchronize()
    want = [t.cpu().clone() for o in outs for t in o] + [nd.cpu().clone()] + [s.cpu().clone() for s in states]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            gouts, gnd = call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in [t for o in gouts for t in o] + [gnd] + states:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [t.cpu() for o in gouts for t in o] + [gnd.cpu()] + [s.cpu() for s in states]
        for i, (a, w) in enumerate(zip(got, want)):
            assert torch.equal(a, w), "replay %d: output %d differs" % (rep, i)
        call()   # eager work between the replays
        torch.cuda.synchronize()
