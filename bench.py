"""Benchmark of the DriftSched admission hot path on one MI355X.

One step = the whole hot path over one batch already resident in HBM:
calibrate (EMA factors from the batch's completion events), characterize
and score (word counts of every prompt, then budgets and classes, fused in
one call: ds_characterize_score; --separate makes them the two calls), and
the dispatch orders of all five policies (ds_order_multi).
Default workload: the largest, 16,384 long-context prompts of 8,192-32,768
words (2.93 GB of packed UTF-8, 5% of the bytes non-ASCII), 16 tenants
(long16k); --workload picks another.

Prints one JSON line: whole-step throughput in requests/s, the roofline of
the dominant stage (characterize + score, HBM-bound) from HIP events recorded
inside the timed steps on the stream the library launches on, and the
single-threaded CPU oracle's throughput on a bounded sample.
The timed steps are eager launches on one stream; --graph times replays of
one step captured in a HIP graph instead (the same launches), and
--schedule overlap runs the stages along their dependencies on two streams
(the FIFO, Priority, Weighted and Aging orders beside calibrate and
characterize + score; SJF after both); both take their stage times from
separate event-instrumented steps.

Inputs: the seeded generator (``workloads``) gives prompts, tenants,
categories, arrivals and each completion event's drift ratio. The events'
admission estimates are the library's own B-free estimates (one ds_score
call with every factor 1, in untimed set-up); the CPU-baseline leg builds
its events the same way with the oracle's score instead.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# rocprofv3 summaries holding the measured HBM bytes of one characterize +
# score call (k_char_main + k_char_fin) in the step, per workload
PROFILES = {"batch64k": os.path.join(ROOT, "profiles", "pipeline_batch64k.md"),
            "long16k": os.path.join(ROOT, "profiles", "pipeline_long16k.md")}
# sources of those two kernels: a summary counts only if taken with them
CHAR_SRCS = [os.path.join(ROOT, "paper_2606_02982_amd", "csrc", f)
             for f in ("characterize.hip", "scoremath.h")]
DEFAULT_WORKLOAD = "long16k"
METRIC = "requests characterized+ordered/sec and achieved HBM GB/s (fraction of peak)"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--stage", choices=["pipeline", "characterize", "errors", "drift", "simulate", "split",
                                        "ceiling", "calibrate"],
                    default="pipeline",
                    help="characterize: time only stage 1 on --workload (any workload with text); "
                         "calibrate: stage 2 alone per call on the completion events of batch4k, "
                         "long16k, batch64k and chat1m, eager and as replays of a captured graph; "
                         "split: Python len(p.split()) per prompt of batch4k on one host core, "
                         "ceiling: the read side of characterize alone over --workload's text size "
                         "(ds_read_bandwidth: the practical read rate of its access pattern); "
                         "the reference point of the paper's tokenizer-overhead table (no GPU); "
                         "errors: the estimation-error diagnostics on --workload's events; "
                         "drift: calibration at each alpha and the Aging re-sorts at every tick "
                         "(drift4m); simulate: the dispatch-tick loop on --workload, per policy")
    ap.add_argument("--settle", type=float, default=0.5,
                    help="seconds of untimed steps before the warmup steps (GPU clocks ramp "
                         "up under sustained load; the timed steps measure the steady state)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run a plain 1 GiB device copy first (to scale memory counters)")
    ap.add_argument("--schedule", choices=["serial", "overlap"], default="serial",
                    help="overlap: stages that do not depend on each other run on two streams "
                         "(calibrate and the budget-free orders beside characterize); serial: "
                         "the four stages one after another on one stream")
    ap.add_argument("--separate", action="store_true",
                    help="stages 1 and 3 as the two calls ds_characterize and ds_score instead of "
                         "the fused ds_characterize_score (the same results)")
    ap.add_argument("--weighted-mode", choices=["blocked", "smooth", "stride"], default="blocked",
                    help="how Weighted interleaves the tiers inside a cycle (ds_order_params."
                         "weighted_mode); the workloads' reading is blocked")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one step captured in a HIP graph instead of eager "
                         "launches (the same kernels)")
    return ap.parse_args()


def to_dev(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    elif a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).cuda()


def bench_split(wl):
    """Python's len(p.split()) on each prompt, one host core: the split() column
    of the paper's tokenizer-overhead comparison, on synthetic prompts."""
    import workloads
    b = workloads.generate(wl.name)
    prompts = [bytes(b.text[b.offsets[i]:b.offsets[i + 1]]).decode("utf-8", "surrogateescape")
               for i in range(b.n)]
    nbytes = int(b.offsets[-1])
    best = None
    for _ in range(3):
        t0 = time.perf_counter()
        counts = [len(p.split()) for p in prompts]
        el = time.perf_counter() - t0
        best = el if best is None or el < best else best
    assert counts == [int(x) for x in b.words], "split() disagrees with the generator's word counts"
    model, nproc = host_cpu()
    print(json.dumps({"metric": "python str.split() per prompt (one host core)", "workload": wl.name,
                      "prompts": b.n, "text_bytes": nbytes, "us_per_prompt": round(best / b.n * 1e6, 3),
                      "MB_per_s": round(nbytes / best / 1e6, 1), "reps": 3, "timing": "best of 3",
                      "host_cores": nproc, "cpu_model": model}), flush=True)


def bench_ceiling(args, wl):
    """ds_read_bandwidth over a buffer of the workload's text size: the same
    wave ranges and loads as characterize, without the classification."""
    import torch
    from paper_2606_02982_amd import driftsched as ds
    import workloads
    nbytes = workloads.generate(wl.name).offsets[-1] // 16 * 16
    buf = torch.randint(0, 256, (int(nbytes),), dtype=torch.uint8, device="cuda")
    out = torch.empty(1, dtype=torch.int32, device="cuda")
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < args.settle:
        ds.read_bandwidth(buf, out)
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        ds.read_bandwidth(buf, out)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        ds.read_bandwidth(buf, out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({"metric": "read side of characterize alone (ds_read_bandwidth) GB/s", "value": round(gbs, 1),
                      "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "ms_per_call": round(ms, 4),
                      "bytes": int(nbytes), "steps": args.steps, "config": {"workload": wl.name}}), flush=True)


def load(wl, with_text=True):
    """The workload's arrays plus its completion events. Each event carries
    its request's B-free admission estimate, taken from one ds_score call
    with every factor 1 (untimed set-up); its observed length is that
    estimate times the event's drift ratio (``workloads.complete``)."""
    import torch
    import workloads
    from paper_2606_02982_amd import driftsched as ds
    b = workloads.generate(wl, with_text=with_text)
    ones = torch.ones(b.n_groups, dtype=torch.float64, device="cuda")
    est_base = ds.score(to_dev(b.words), to_dev(b.category), to_dev(b.tenant), to_dev(b.group),
                        to_dev(b.t_base), to_dev(b.s_tenant), ones, f_ref=b.f_ref)[0]
    return workloads.complete(b, est_base.cpu().numpy())


def oracle_events(b):
    """A copy of batch b whose completion events are built from the oracle's
    own score (the CPU-baseline leg takes no input from the GPU)."""
    import oracle
    import workloads
    c = workloads.Batch(b)
    est_base = oracle.score(b.words, b.category, b.tenant, b.group, b.t_base, b.s_tenant,
                            np.ones(b.n_groups), f_ref=b.f_ref)[0]
    return workloads.complete(c, est_base)


def host_cpu():
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count()


def main():
    args = parse()
    if args.stage == "split":
        import workloads
        return bench_split(workloads.WORKLOADS["batch4k"])
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: the admission hot path runs on one GPU here; --gpus %d is not "
              "supported (how the path would shard is described in the documentation)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    from paper_2606_02982_amd import driftsched as ds

    torch.cuda.set_device(0)
    wl = workloads.WORKLOADS[args.workload]
    if args.stage == "characterize":
        return bench_characterize(args, wl)
    if args.stage == "ceiling":
        return bench_ceiling(args, wl)
    if args.stage == "errors":
        return bench_errors(args, wl)
    if args.stage == "drift":
        return bench_drift(args, workloads.WORKLOADS["drift4m"] if wl.has_text else wl)
    if args.stage == "simulate":
        return bench_simulate(args, wl)
    if args.stage == "calibrate":
        return bench_calibrate(args)
    if not wl.has_text or len(wl.policies) < 5:
        print("bench.py: the step needs a workload with text and all five policies", file=sys.stderr)
        sys.exit(2)
    t0 = time.time()
    b = load(wl)
    gen_s = time.time() - t0
    N = b.n
    B = len(b.text)
    print("bench: workload %s, %d requests, %d text bytes (generated in %.1fs)" % (
        wl.name, N, B, gen_s), file=sys.stderr, flush=True)

    if args.copy_probe:
        copy_probe()

    # device-resident inputs
    text, offsets = to_dev(b.text), to_dev(b.offsets)
    ev_group, ev_est, ev_obs = to_dev(b.ev_group), to_dev(b.ev_est), to_dev(b.ev_obs)
    category, tenant, group = to_dev(b.category), to_dev(b.tenant), to_dev(b.group)
    t_base, s_tenant = to_dev(b.t_base), to_dev(b.s_tenant)
    tier, arrival = to_dev(b.tier), to_dev(b.arrival)
    state = torch.ones(b.n_groups, dtype=torch.float64, device="cuda")
    # outputs
    counts = torch.empty(N, dtype=torch.int32, device="cuda")
    trace = torch.empty(N, dtype=torch.float64, device="cuda")
    sc_out = (torch.empty(N, dtype=torch.float64, device="cuda"),
              torch.empty(N, dtype=torch.float64, device="cuda"),
              torch.empty(N, dtype=torch.float64, device="cuda"),
              torch.empty(N, dtype=torch.uint8, device="cuda"))
    perms = [torch.empty(N, dtype=torch.int32, device="cuda") for _ in range(5)]
    params = ds.order_params(weights=tuple(int(w) for w in b.weights),
                             tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate,
                             t_now=b.t_now, aging_floor=b.aging_floor, weighted_mode=args.weighted_mode)
    ws = {op: ds.workspace(op, N, b.n_groups) for op in range(5)}
    ALL = (0, 1, 2, 3, 4)
    perm_map = dict(enumerate(perms))
    alpha = b.alphas[0]
    torch.cuda.synchronize()

    def char_score():
        """Stages 1 and 3: one fused call, or the two calls (--separate)."""
        if args.separate:
            ds.characterize(text, offsets, counts=counts, ws=ws[ds.OP_CHARACTERIZE])
            ds.score(counts, category, tenant, group, t_base, s_tenant, state, out=sc_out)
        else:
            ds.characterize_score(text, offsets, category, tenant, group, t_base, s_tenant, state,
                                  counts=counts, out=sc_out, ws=ws[ds.OP_CHARACTERIZE])

    def step(ev=None):
        """The stages one after another on the current stream (the one the
        library launches on): calibrate (its factors are final before
        scoring), characterize + score, the five orders. ev: four events
        recorded between the stages."""
        if ev: ev[0].record()
        ds.calibrate(ev_group, ev_est, ev_obs, alpha, state, trace=trace, ws=ws[ds.OP_CALIBRATE])
        if ev: ev[1].record()
        char_score()
        if ev: ev[2].record()
        ds.order_multi(ALL, tier, arrival, sc_out[2], params=params, perms=perm_map,
                       ws=ws[ds.OP_ORDER_MULTI])
        if ev: ev[3].record()

    # The same work along the stages' dependencies: FIFO, Priority, Weighted
    # and Aging read only tiers and arrivals, so they run on a second stream
    # beside calibrate and characterize + score; SJF (budget-keyed) follows
    # both and reuses the FIFO permutation.
    aux = torch.cuda.Stream()
    ws_aux = ds.workspace(ds.OP_ORDER_MULTI, N, b.n_groups)
    budget = sc_out[2]

    def step_overlap():
        main_s = torch.cuda.current_stream()
        aux.wait_stream(main_s)
        with torch.cuda.stream(aux):
            ds.order_multi((0, 1, 2, 4), tier, arrival, params=params, perms=perm_map, ws=ws_aux)
        ds.calibrate(ev_group, ev_est, ev_obs, alpha, state, trace=trace, ws=ws[ds.OP_CALIBRATE])
        char_score()
        main_s.wait_stream(aux)
        ds.order_multi((3,), tier, arrival, budget, fifo=perms[0], params=params, perms=perm_map,
                       ws=ws[ds.OP_ORDER_MULTI])

    plain = args.schedule == "serial" and not args.graph
    run = step if args.schedule == "serial" else step_overlap

    settle(run, args.settle)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    if not plain:
        # stage times from serial steps with events between the stages
        for k in range(args.steps):
            step(evs[k])
        torch.cuda.synchronize()
    serial_out = [perms[i].clone() for i in (0, 1, 2, 4)] + [counts.clone()]
    # the timed region: K steps of the timed schedule; with the plain serial
    # schedule the stage events are recorded inside it
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        if plain:
            step(evs[k])
        else:
            run()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_eager = wall * 1e3 / args.steps
    for a, b_ in zip(serial_out, [perms[i] for i in (0, 1, 2, 4)] + [counts]):
        assert torch.equal(a, b_), "the %s schedule differs from the serial step" % args.schedule

    if args.graph:
        # the whole step (every launch of the four stages) captured once in a
        # HIP graph and replayed; the step time is the replays'. The replays'
        # outputs must equal the eager step's.
        # (the factors keep folding the same events step after step, so the
        # budgets and the SJF order may move by rounding; the others may not)
        eager = [perms[i].clone() for i in (0, 1, 2, 4)] + [counts.clone()]
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            run()
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=cap):
                run()
        torch.cuda.current_stream().wait_stream(cap)
        torch.cuda.synchronize()
        settle(g.replay, args.settle)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        for a, b_ in zip(eager, [perms[i] for i in (0, 1, 2, 4)] + [counts]):
            assert torch.equal(a, b_), "graph replay differs from the eager step"

    stage_ms = np.zeros(3)
    for e in evs:
        for s in range(3):
            stage_ms[s] += e[s].elapsed_time(e[s + 1])
    stage_ms /= args.steps
    ms_per_step = wall * 1e3 / args.steps
    value = N * args.steps / wall

    # algorithmic bytes (what the method must move) per stage
    char_bytes = B + 8 * (N + 1) + 4 * N
    cal_bytes = 16 * N + 8 * N + 16 * b.n_groups
    # score: category, tenant, group read; est_base, est, budget, class
    # written (the two separate calls read the counts back as well)
    score_bytes = (1 + 4 + 4) * N + (8 + 8 + 8 + 1) * N + (4 * N if args.separate else 0)
    order_bytes = (12 + 13 + 13 + 20 + 13) * N
    cs_bytes = char_bytes + score_bytes
    char_gbs = cs_bytes / (stage_ms[1] * 1e-3) / 1e9
    total_gbs = (char_bytes + cal_bytes + score_bytes + order_bytes) / (ms_per_step * 1e-3) / 1e9

    # sanity: the counts of the last step equal the generator's word counts
    assert np.array_equal(counts.cpu().numpy().view(np.uint32), b.words), "counts mismatch"

    # the practical read ceiling of characterize's access pattern, after the
    # timed region: its read side alone over the same text buffer
    rb = (int(text.numel()) // 16) * 16
    rbuf, rout = text[:rb], torch.empty(ds.READ_BW_WORDS, dtype=torch.int32, device="cuda")
    for _ in range(5):
        ds.read_bandwidth(rbuf, rout)
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    r0.record()
    for _ in range(20):
        ds.read_bandwidth(rbuf, rout)
    r1.record()
    torch.cuda.synchronize()
    ceil_gbs = rb / (r0.elapsed_time(r1) / 20 * 1e-3) / 1e9

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(oracle_events(b), args.cpu_seconds, args.weighted_mode)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_s": args.settle,
        "graph": bool(args.graph),
        "schedule": args.schedule,
        "ms_per_step_eager": round(ms_eager, 4),
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8+f64",
        "data": "synthetic",
        "config": {"workload": wl.name, "requests": N, "text_bytes": B, "tenants": b.n_groups,
                   "events": N, "policies": 5, "description": wl.note},
        "hbm_gbs_step": round(total_gbs, 1),
        "hbm_frac_step": round(total_gbs / HBM_PEAK_GBS, 4),
        "stages_ms": {"calibrate": round(stage_ms[0], 4), "characterize_score": round(stage_ms[1], 4),
                      "order_x5": round(stage_ms[2], 4)},
        "stage_events": "inside the timed steps" if plain else "separate serial steps",
        "fused_characterize_score": not args.separate,
        "weighted_mode": args.weighted_mode,
        "roofline": {"kernel": "characterize + score (k_char_main + k_char_fin)" if not args.separate
                     else "characterize + score (k_char_main + k_char_fin, k_score)",
                     "bound": "hbm", "achieved": round(char_gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(char_gbs / HBM_PEAK_GBS, 4),
                     "avg_launch_ms": round(stage_ms[1], 4),
                     "algorithmic_bytes": int(cs_bytes),
                     "traffic": None if args.separate else measured_traffic(wl.name)},
        "cpu_baseline": cpu,
        "read_ceiling": {"kernel": "ds_read_bandwidth (characterize's waves and loads, no classification)",
                         "achieved": round(ceil_gbs, 1), "unit": "GB/s", "frac": round(ceil_gbs / HBM_PEAK_GBS, 4),
                         "characterize_score_of_ceiling": round(char_gbs / ceil_gbs, 4)},
    }
    print(json.dumps(out), flush=True)


def settle(fn, seconds):
    """Untimed repetitions of fn for about `seconds` of wall time."""
    import torch
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            fn()
        torch.cuda.synchronize()


def copy_probe():
    """A plain 1 GiB device copy: the reference reading of the memory counters."""
    import torch
    x = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    del x, y


def bench_characterize(args, wl):
    """Stage 1 alone on one workload: HBM roofline of the word counter."""
    import torch
    from paper_2606_02982_amd import driftsched as ds
    import workloads
    b = workloads.generate(wl)
    N, B = b.n, len(b.text)
    if args.copy_probe:
        copy_probe()
    text, offsets = to_dev(b.text), to_dev(b.offsets)
    counts = torch.empty(N, dtype=torch.int32, device="cuda")
    ws = ds.workspace(ds.OP_CHARACTERIZE, N)
    call = lambda: ds.characterize(text, offsets, counts=counts, ws=ws)
    settle(call, args.settle)
    for _ in range(args.warmup):
        call()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(args.steps):
        ds.characterize(text, offsets, counts=counts, ws=ws)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / args.steps
    assert np.array_equal(counts.cpu().numpy().view(np.uint32), b.words), "counts mismatch"
    nbytes = B + 8 * (N + 1) + 4 * N
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({"metric": "characterize HBM GB/s", "value": round(gbs, 1), "unit": "GB/s",
                      "frac": round(gbs / HBM_PEAK_GBS, 4), "ms_per_call": round(ms, 4),
                      "algorithmic_bytes": int(nbytes),
                      "requests_per_s": round(N / (ms * 1e-3), 1), "steps": args.steps,
                      "config": {"workload": wl.name, "requests": N, "text_bytes": B,
                                 "nonascii_byte_frac": round(float((b.text >= 0x80).mean()), 4)}}),
          flush=True)


def bench_errors(args, wl):
    """The evaluation diagnostics on one workload's completion events: error
    statistics with and without the calibrated factor, and the class histogram
    of the batch (HBM-bound reductions)."""
    import torch
    from paper_2606_02982_amd import driftsched as ds
    b = load(wl, with_text=False)
    E, G = len(b.ev_group), b.n_groups
    group, est, obs = to_dev(b.ev_group), to_dev(b.ev_est), to_dev(b.ev_obs)
    state = torch.ones(G, dtype=torch.float64, device="cuda")
    before = torch.empty(E, dtype=torch.float64, device="cuda")
    ds.calibrate(group, est, obs, b.alphas[0], state, trace=False, trace_before=before)
    cat = to_dev(b.category)
    cls = to_dev(np.minimum(b.words % 3, 2).astype(np.uint8))   # any class values serve
    out = torch.empty((G + 1, 4), dtype=torch.float64, device="cuda")
    hist = torch.empty((len(b.t_base), 3), dtype=torch.int32, device="cuda")
    ws = ds.workspace(ds.OP_ERROR_STATS, E, G)

    def timed(fn):
        settle(fn, args.settle)
        for _ in range(args.warmup):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(args.steps):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / args.steps

    ms_off = timed(lambda: ds.error_stats(est, obs, group=group, n_groups=G, out=out, ws=ws))
    ms_on = timed(lambda: ds.error_stats(est, obs, factor=before, group=group, n_groups=G, out=out,
                                         ws=ws))
    ms_hist = timed(lambda: ds.class_histogram(cat, cls, len(b.t_base), out=hist))
    bytes_off = E * (8 + 4 + 4) + (G + 1) * 32
    bytes_on = bytes_off + E * 8
    bytes_hist = b.n * 2 + len(b.t_base) * 12
    res = {"metric": "evaluation diagnostics HBM GB/s", "unit": "GB/s",
           "config": {"workload": wl.name, "events": E, "groups": G, "requests": b.n},
           "error_stats_bias_off": {"ms": round(ms_off, 4), "GBs": round(bytes_off / ms_off / 1e6, 1)},
           "error_stats_bias_on": {"ms": round(ms_on, 4), "GBs": round(bytes_on / ms_on / 1e6, 1)},
           "class_histogram": {"ms": round(ms_hist, 4), "GBs": round(bytes_hist / ms_hist / 1e6, 1)},
           "peak": HBM_PEAK_GBS}
    print(json.dumps(res), flush=True)


def timed_ms(fn, args):
    """Mean milliseconds per call of fn over args.steps calls after the settle
    and warmup calls (HIP events on torch's current stream, where the library
    launches)."""
    import torch
    settle(fn, args.settle)
    for _ in range(args.warmup):
        fn()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(args.steps):
        fn()
    ev[1].record()
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / args.steps


def bench_calibrate(args):
    """Stage 2 alone on each workload's completion events: microseconds per
    call, eager (HIP events around args.steps calls) and as replays of a
    graph capturing 20 calls (no host launch gaps), with the final factors of
    one call from 1.0 checked against the oracle."""
    import torch
    import oracle
    import workloads
    from paper_2606_02982_amd import driftsched as ds
    res = {"metric": "calibration microseconds per call (stage 2 alone)", "steps": args.steps,
           "workloads": {}}
    for name in ("batch4k", "long16k", "batch64k", "chat1m"):
        b = load(workloads.WORKLOADS[name], with_text=False)
        ob = oracle_events(b)
        E, G = len(b.ev_group), b.n_groups
        group, est, obs = to_dev(b.ev_group), to_dev(b.ev_est), to_dev(b.ev_obs)
        state = torch.ones(G, dtype=torch.float64, device="cuda")
        trace = torch.empty(E, dtype=torch.float64, device="cuda")
        ws = ds.workspace(ds.OP_CALIBRATE, E, G)
        alpha = b.alphas[0]

        def cal():
            ds.calibrate(group, est, obs, alpha, state, trace=trace, ws=ws)
        eager_ms = timed_ms(cal, args)
        k = 20
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            cal()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                for _ in range(k):
                    cal()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph_ms = timed_ms(g.replay, args) / k
        state.fill_(1.0)
        cal()
        want, _ = oracle.calibrate(ob.ev_group, ob.ev_est, ob.ev_obs, alpha, np.ones(G))
        assert np.all(np.abs(state.cpu().numpy() - want) <= 1e-12 * np.abs(want)), "calibration mismatch"
        cal_bytes = E * (4 + 8 + 4) + E * 8 + 16 * G
        res["workloads"][name] = {"events": E, "groups": G, "us_per_call_eager": round(eager_ms * 1e3, 2),
                                  "us_per_call_graph": round(graph_ms * 1e3, 2),
                                  "GBs_graph": round(cal_bytes / (graph_ms * 1e-3) / 1e9, 1)}
    print(json.dumps(res))


def bench_drift(args, wl):
    """The drift workload: 4,194,304 completion events over 4,096 tenants
    folded into the calibration factors at each alpha (events/s), and the
    Aging order of the pending set recomputed at each of the 64 ticks (keys
    re-sorted/s). Requests are stored in arrival order, so the pending set of
    tick k is the first n_k requests and its FIFO order is the first n_k
    entries of the whole set's FIFO order."""
    import torch
    import oracle
    from paper_2606_02982_amd import driftsched as ds
    b = load(wl)
    ob = oracle_events(b)
    if args.copy_probe:
        copy_probe()
    E, G = len(b.ev_group), b.n_groups
    group, est, obs = to_dev(b.ev_group), to_dev(b.ev_est), to_dev(b.ev_obs)
    state = torch.ones(G, dtype=torch.float64, device="cuda")
    trace = torch.empty(E, dtype=torch.float64, device="cuda")
    ws_cal = ds.workspace(ds.OP_CALIBRATE, E, G)
    res = {"metric": "drift workload: calibration events/s and Aging keys re-sorted/s",
           "config": {"workload": wl.name, "events": E, "groups": G, "ticks": len(b.tick_t),
                      "keys_over_ticks": int(b.tick_n.sum()), "alphas": list(wl.alphas)},
           "steps": args.steps, "peak_GBs": HBM_PEAK_GBS}
    cal_bytes = E * (4 + 8 + 4) + E * 8 + 16 * G
    for alpha in wl.alphas:
        def cal():
            ds.calibrate(group, est, obs, alpha, state, trace=trace, ws=ws_cal)
        ms = timed_ms(cal, args)
        # parity of the final factors after one call from 1.0
        state.fill_(1.0)
        cal()
        want, _ = oracle.calibrate(ob.ev_group, ob.ev_est, ob.ev_obs, alpha, np.ones(G))
        got = state.cpu().numpy()
        assert np.all(np.abs(got - want) <= 1e-12 * np.abs(want)), "calibration mismatch"
        res["calibrate_alpha_%g" % alpha] = {
            "ms": round(ms, 4), "events_per_s": round(E / (ms * 1e-3), 1),
            "GBs": round(cal_bytes / (ms * 1e-3) / 1e9, 1)}

    tier, arrival = to_dev(b.tier), to_dev(b.arrival)
    N = b.n
    fifo_full, _ = ds.order(ds.FIFO, tier, arrival)
    perm = torch.empty(N, dtype=torch.int32, device="cuda")
    perm_fifo = torch.empty(N, dtype=torch.int32, device="cuda")
    ws_o = ds.workspace(ds.OP_ORDER_MULTI, N)
    kw = dict(weights=tuple(int(w) for w in b.weights), tier_priority=tuple(b.tier_priority),
              aging_rate=b.aging_rate, aging_floor=b.aging_floor)
    ticks = [(int(nk), ds.order_params(t_now=float(t), **kw)) for nk, t in zip(b.tick_n, b.tick_t)]
    total = int(b.tick_n.sum())

    def aging_ticks():
        for nk, p in ticks:
            ds.order(ds.AGING, tier[:nk], arrival[:nk], fifo=fifo_full[:nk], params=p,
                     perm=perm[:nk], ws=ws_o)

    def aging_ticks_with_fifo():
        for nk, p in ticks:
            ds.order_multi((ds.FIFO, ds.AGING), tier[:nk], arrival[:nk], params=p,
                           perms={ds.FIFO: perm_fifo[:nk], ds.AGING: perm[:nk]}, ws=ws_o)

    steps = max(1, args.steps // 10)
    a2 = argparse.Namespace(**dict(vars(args), steps=steps, warmup=1))
    ms = timed_ms(aging_ticks, a2)
    ms_f = timed_ms(aging_ticks_with_fifo, a2)
    # parity of the first tick's order
    n1, p1 = ticks[0]
    got, _ = ds.order(ds.AGING, tier[:n1], arrival[:n1], fifo=fifo_full[:n1], params=p1)
    want, _ = oracle.order(4, b.tier[:n1], b.arrival[:n1], None, t_now=float(b.tick_t[0]), **kw)
    assert np.array_equal(got.cpu().numpy().view(np.uint32), want), "aging order mismatch"
    res["aging_64_ticks"] = {"ms": round(ms, 4), "keys_per_s": round(total / (ms * 1e-3), 1),
                             "ms_with_fifo_sort": round(ms_f, 4),
                             "keys_per_s_with_fifo_sort": round(total / (ms_f * 1e-3), 1),
                             "GBs": round(13 * total / (ms * 1e-3) / 1e9, 1)}
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        oracle.calibrate(ob.ev_group, ob.ev_est, ob.ev_obs, wl.alphas[0], np.ones(G))
        cal_s = time.perf_counter() - t0
        t0 = time.perf_counter()
        done = 0
        for k, (nk, p) in enumerate(ticks):
            oracle.order(4, b.tier[:nk], b.arrival[:nk], None, t_now=float(b.tick_t[k]), **kw)
            done += nk
            if time.perf_counter() - t0 > args.cpu_seconds:
                break
        ag_s = time.perf_counter() - t0
        res["cpu_baseline"] = {"calibrate_events_per_s": round(E / cal_s, 1),
                               "aging_keys_per_s": round(done / ag_s, 1), "cores": 1,
                               "kind": "oracle",
                               "sample": "one calibration pass over all events; Aging orders "
                                         "of the first %d ticks (%d keys, %.1f s)" % (k + 1, done, ag_s)}
    print(json.dumps(res), flush=True)


def bench_simulate(args, wl):
    """The dispatch-tick loop over one workload's requests for each policy:
    10 ms ticks dispatching batches of 32, completions folded into the
    factors between ticks. Reports ticks/s and requests dispatched/s."""
    import torch
    from paper_2606_02982_amd import driftsched as ds
    import workloads
    b = load(wl, with_text=False)
    ticks = workloads.sim_ticks(b.arrival)
    d = {k: to_dev(getattr(b, k)) for k in ("arrival", "tier", "words", "category", "tenant",
                                            "group", "observed", "t_base", "s_tenant")}
    tick_t = to_dev(ticks)
    state = torch.ones(b.n_groups, dtype=torch.float64, device="cuda")
    N = b.n
    out = (torch.empty(N, dtype=torch.int32, device="cuda"),
           torch.empty(N, dtype=torch.int32, device="cuda"),
           torch.empty(1, dtype=torch.int32, device="cuda"))
    ws = ds.workspace(ds.OP_SIMULATE, N)
    res = {"metric": "dispatch-tick loop: ticks/s and requests dispatched/s",
           "config": {"workload": wl.name, "requests": N, "ticks": len(ticks), "batch": 32,
                      "tick_s": 0.01}, "policies": {}}
    steps = max(1, args.steps // 10)
    a2 = argparse.Namespace(**dict(vars(args), steps=steps, warmup=1, settle=0.0))
    # every policy (and the other two Weighted interleavings) in one launch
    kw = dict(alpha=b.alphas[0], weights=tuple(int(w) for w in b.weights),
              tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate)
    runs = [(name, pol, "blocked") for name, pol in ds.POLICIES.items()] + \
        [("weighted_smooth", ds.WEIGHTED, "smooth"), ("weighted_stride", ds.WEIGHTED, "stride")]
    mparams = [ds.sim_params(pol, batch=32, weighted_mode=m, **kw) for _, pol, m in runs]
    mstates = [torch.ones(b.n_groups, dtype=torch.float64, device="cuda") for _ in runs]
    mws = ds.workspace(ds.OP_SIMULATE_MULTI, N, len(runs))

    def run_multi():
        for st in mstates:
            st.fill_(1.0)
        return ds.simulate_multi(d["arrival"], d["tier"], d["words"], d["category"], d["tenant"],
                                 d["group"], d["observed"], d["t_base"], d["s_tenant"], mstates, tick_t,
                                 mparams, ws=mws)
    ms_multi = timed_ms(run_multi, a2)
    _, nd_multi = run_multi()
    res["one_launch"] = {"runs": [r[0] for r in runs], "ms": round(ms_multi, 3),
                         "dispatched": [int(x) for x in nd_multi.cpu()],
                         "ticks_per_s_per_run": round(len(ticks) / (ms_multi * 1e-3), 1)}
    # a sweep that fills the GPU (one workgroup per run, up to one per CU):
    # the five policies in turn at EMA weights spread over [0.02, 0.5], as
    # many runs as ds.SIM_MAX_RUNS allows within a 48 GB workspace
    per_run = ds.workspace_bytes(ds.OP_SIMULATE_MULTI, N, 2) - ds.workspace_bytes(ds.OP_SIMULATE_MULTI, N, 1)
    R = int(min(ds.SIM_MAX_RUNS, max(8, (48 << 30) // max(per_run, 1))))
    pols = list(ds.POLICIES.values())
    sweep_alpha = [0.02 + 0.48 * (r // 5) / max(1, (R - 1) // 5) for r in range(R)]
    kw_sweep = {k: v for k, v in kw.items() if k != "alpha"}
    sweep = [ds.sim_params(pols[r % 5], batch=32, alpha=sweep_alpha[r], **kw_sweep) for r in range(R)]
    sstates = [torch.ones(b.n_groups, dtype=torch.float64, device="cuda") for _ in range(R)]
    sws = ds.workspace(ds.OP_SIMULATE_MULTI, N, R)

    def run_sweep():
        for st in sstates:
            st.fill_(1.0)
        return ds.simulate_multi(d["arrival"], d["tier"], d["words"], d["category"], d["tenant"],
                                 d["group"], d["observed"], d["t_base"], d["s_tenant"], sstates, tick_t,
                                 sweep, ws=sws)
    ms_sweep = timed_ms(run_sweep, a2)
    _, nd_sweep = run_sweep()
    tot = int(nd_sweep.to(torch.int64).sum().cpu())
    res["sweep"] = {"runs": R, "policies": "the five in turn", "alphas": [round(sweep_alpha[0], 4),
                                                                          round(sweep_alpha[-1], 4)],
                    "ms": round(ms_sweep, 3), "dispatched_total": tot,
                    "requests_per_s": round(tot / (ms_sweep * 1e-3), 1),
                    "ticks_per_s_per_run": round(len(ticks) / (ms_sweep * 1e-3), 1)}
    del sws, sstates
    for name, pol in ds.POLICIES.items():
        p = ds.sim_params(pol, batch=32, alpha=b.alphas[0], weights=tuple(int(w) for w in b.weights),
                          tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate,
                          weighted_mode=args.weighted_mode)

        def run():
            state.fill_(1.0)
            ds.simulate(d["arrival"], d["tier"], d["words"], d["category"], d["tenant"], d["group"],
                        d["observed"], d["t_base"], d["s_tenant"], state, tick_t, p, out=out, ws=ws)
        ms = timed_ms(run, a2)
        nd = int(out[2].cpu()[0])
        res["policies"][name] = {"ms": round(ms, 3), "ticks_per_s": round(len(ticks) / (ms * 1e-3), 1),
                                 "dispatched": nd,
                                 "requests_per_s": round(nd / (ms * 1e-3), 1)}
    print(json.dumps(res), flush=True)


def measured_traffic(workload):
    """HBM bytes per characterize + score call (k_char_main + k_char_fin) from
    the committed rocprofv3 counter summary of this workload's step, if it was
    taken with the current kernel sources."""
    import hashlib
    path = PROFILES.get(workload)
    if path is None or not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip() in ("traffic_bytes_per_call",
                                                          "characterize_source_sha256_16"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in CHAR_SRCS:
        h.update(open(f, "rb").read())
    sha = h.hexdigest()[:16]
    if vals.get("characterize_source_sha256_16") != sha or "traffic_bytes_per_call" not in vals:
        return None
    return int(vals["traffic_bytes_per_call"])


def cpu_baseline(b, budget_s, weighted_mode="blocked"):
    """The oracle as it stands, single-threaded, on the same step.

    Stage 1 is timed on the batch's prompts in order until about half of
    ``budget_s`` has passed (a bounded sample of the same text), the other
    stages on the whole batch; the step time per request is the sample's
    stage-1 time per prompt plus the other stages' time per request."""
    import oracle
    N = b.n
    kw = dict(weights=tuple(int(w) for w in b.weights), tier_priority=tuple(b.tier_priority),
              aging_rate=b.aging_rate, t_now=b.t_now, aging_floor=b.aging_floor)
    # stage 1 on a prefix of the prompts, in chunks
    done, t_char, chunk = 0, 0.0, 64
    while done < N and t_char < 0.5 * budget_s:
        k = min(chunk, N - done)
        lo, hi = int(b.offsets[done]), int(b.offsets[done + k])
        sub_off = b.offsets[done:done + k + 1] - b.offsets[done]
        t0 = time.perf_counter()
        got = oracle.characterize(b.text[lo:hi], sub_off)
        t_char += time.perf_counter() - t0
        assert np.array_equal(got, b.words[done:done + k]), "oracle counts differ from the generator's"
        done += k
        chunk = min(chunk * 2, 1 << 16)
    sample_bytes = int(b.offsets[done])
    # the other stages on the whole batch (the counts are the generator's, which
    # stage 1 reproduces exactly)
    t = [time.perf_counter()]
    state, _ = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, b.alphas[0], np.ones(b.n_groups))
    t.append(time.perf_counter())
    _, _, budget, _ = oracle.score(b.words, b.category, b.tenant, b.group, b.t_base,
                                   b.s_tenant, state)
    t.append(time.perf_counter())
    weighted = {"blocked": 2, "smooth": oracle.WEIGHTED_SMOOTH, "stride": oracle.WEIGHTED_STRIDE}
    for pol in (0, 1, weighted[weighted_mode], 3, 4):
        oracle.order(pol, b.tier, b.arrival, budget, **kw)
        t.append(time.perf_counter())
    t_rest = t[-1] - t[0]
    per_req = t_char / done + t_rest / N
    model, nproc = host_cpu()
    stage_s = {"characterize": t_char / done * N, "calibrate": t[1] - t[0], "score": t[2] - t[1]}
    for k, name in enumerate(("fifo", "priority", "weighted", "sjf", "aging")):
        stage_s["order_" + name] = t[3 + k] - t[2 + k]
    return {"value": round(1.0 / per_req, 1), "unit": "requests/s", "cores": 1, "kind": "oracle",
            "host_cpu": model, "host_nproc": nproc,
            "sample": "stage 1 on the first %d of %d prompts (%d bytes, %.1f s); calibrate, score "
                      "and the five orders on the whole batch (%.1f s); step time per request = "
                      "the sum of the two per-request times" % (done, N, sample_bytes, t_char, t_rest),
            "stage1_MB_per_s": round(sample_bytes / t_char / 1e6, 1),
            "stage_s": {k: round(v, 6) for k, v in stage_s.items()}}


if __name__ == "__main__":
    main()
