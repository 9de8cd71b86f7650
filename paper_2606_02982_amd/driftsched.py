"""Python binding of the DriftSched C ABI (include/driftsched.h).

Argument marshalling only: every step runs in the HIP library
``libdriftsched.so``. Arrays are torch tensors on the current HIP device;
work is enqueued on torch's current stream. Unsigned 32-bit arrays travel as
torch.int32 and uint64 offsets as torch.int64 (same bits for the values the
library accepts).

The library must be built (``paper_2606_02982_amd.build.build()``); without
it importing this module fails. There is no fallback.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdriftsched.so")

FIFO, PRIORITY, WEIGHTED, SJF, AGING = 0, 1, 2, 3, 4
POLICIES = {"fifo": FIFO, "priority": PRIORITY, "weighted": WEIGHTED, "sjf": SJF, "aging": AGING}
OP_CHARACTERIZE, OP_CALIBRATE, OP_SCORE, OP_ORDER, OP_ORDER_MULTI = 0, 1, 2, 3, 4
OP_ERROR_STATS, OP_CLASS_HIST, OP_SIMULATE, OP_SIMULATE_MULTI = 5, 6, 7, 8
SIM_MAX_RUNS = 256
DS_VALIDATE = 1
DS_SERIAL_SORT = 2
DS_NO_WAIT = 4          # diagnostic: bounded device-side waits give up at once
ERR_WAIT = -8           # DS_ERR_WAIT
WS_STATUS_OFFSET = 4    # byte offset of the bounded-wait status word in a workspace
MAX_TIERS = 16
WRR_BLOCKED, WRR_SMOOTH, WRR_STRIDE = 0, 1, 2   # ds_order_params.weighted_mode
WRR_MAX_WEIGHT_SUM = 1024
MAX_BATCH = 1024


class DriftSchedError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s (status %d)" % (msg, status))
        self.status = status


class ScoreParams(ctypes.Structure):
    _fields_ = [("f_ref", ctypes.c_double), ("short_max", ctypes.c_double),
                ("medium_max", ctypes.c_double)]


class OrderParams(ctypes.Structure):
    _fields_ = [("n_tiers", ctypes.c_uint32), ("weight", ctypes.c_uint32 * MAX_TIERS),
                ("tier_priority", ctypes.c_double * MAX_TIERS), ("aging_rate", ctypes.c_double),
                ("t_now", ctypes.c_double), ("aging_floor", ctypes.c_double),
                ("weighted_mode", ctypes.c_uint32)]


class SimParams(ctypes.Structure):
    _fields_ = [("policy", ctypes.c_int), ("batch", ctypes.c_uint32), ("alpha", ctypes.c_double),
                ("score", ScoreParams), ("order", OrderParams)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libdriftsched.so is not built (run paper_2606_02982_amd.build.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, u32, u64, f64, i32 = (ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64,
                             ctypes.c_double, ctypes.c_int)
    sz = ctypes.c_size_t
    lib.ds_characterize.argtypes = [P, u64, P, u32, P, P, sz, u32, P]
    lib.ds_calibrate.argtypes = [P, P, P, u64, f64, u32, P, P, P, sz, u32, P]
    lib.ds_calibrate_ex.argtypes = [P, P, P, u64, f64, u32, P, P, P, P, sz, u32, P]
    lib.ds_error_stats.argtypes = [u64, P, P, P, P, u32, P, P, sz, u32, P]
    lib.ds_class_histogram.argtypes = [u32, P, u32, P, P, P, sz, u32, P]
    lib.ds_read_bandwidth.argtypes = [P, u64, P, P]
    lib.ds_score.argtypes = [u32, P, P, P, P, P, u32, P, u32, P, u32, ctypes.POINTER(ScoreParams),
                             P, P, P, P, P, sz, u32, P]
    lib.ds_characterize_score.argtypes = [P, u64, P, u32, P, P, P, P, P, u32, P, u32, P, u32,
                                          ctypes.POINTER(ScoreParams), P, P, P, P, P, sz, u32, P]
    lib.ds_characterize_score_noalloc.argtypes = [P, u64, P, u32, P, P, P, P, P, u32, P, u32, P, u32,
                                                  ctypes.POINTER(ScoreParams), P, P, P, P, u32, P]
    lib.ds_order.argtypes = [i32, u32, P, P, P, P, ctypes.POINTER(OrderParams), P, P, P, sz, u32, P]
    lib.ds_order_multi.argtypes = [u32, u32, P, P, P, P, ctypes.POINTER(OrderParams),
                                   ctypes.POINTER(P), ctypes.POINTER(P), P, sz, u32, P]
    lib.ds_simulate.argtypes = [u32, P, P, P, P, P, P, P, P, u32, P, u32, u32, P, u32,
                                ctypes.POINTER(SimParams), P, P, P, P, P, sz, u32, P]
    lib.ds_simulate_multi.argtypes = [u32, u32, P, P, P, P, P, P, P, P, u32, P, u32, u32, P, u32,
                                      ctypes.POINTER(SimParams), ctypes.POINTER(P), ctypes.POINTER(P),
                                      ctypes.POINTER(P), P, P, sz, u32, P]
    for f in (lib.ds_characterize, lib.ds_characterize_score, lib.ds_characterize_score_noalloc,
              lib.ds_calibrate, lib.ds_calibrate_ex, lib.ds_score, lib.ds_order,
              lib.ds_order_multi, lib.ds_error_stats, lib.ds_class_histogram, lib.ds_simulate,
              lib.ds_simulate_multi):
        f.restype = i32
    lib.ds_workspace_bytes.argtypes = [i32, u64, u32]
    lib.ds_workspace_bytes.restype = sz
    lib.ds_status_string.argtypes = [i32]
    lib.ds_status_string.restype = ctypes.c_char_p
    lib.ds_version.argtypes = []
    lib.ds_version.restype = u32
    return lib


lib = _load()

_ws_cache = {}


def status_string(status):
    return lib.ds_status_string(int(status)).decode()


def workspace_bytes(op, n, n_groups=0):
    return int(lib.ds_workspace_bytes(int(op), int(n), int(n_groups)))


def workspace(op, n, n_groups=0, device=None):
    """Cached device workspace (uint8 tensor) big enough for op at size n."""
    device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
    need = max(workspace_bytes(op, n, n_groups), 256)
    key = (device.index, op)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < need:
        buf = torch.empty(need, dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    return buf


def _check(status):
    if status != 0:
        raise DriftSchedError(status, status_string(status))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _flags(validate, no_wait=False):
    return (DS_VALIDATE if validate else 0) | (DS_NO_WAIT if no_wait else 0)


def wait_status(ws):
    """The bounded-wait status word of a workspace after a call (0: no wait
    ran out). Synchronizes with the current stream."""
    return int(ws[WS_STATUS_OFFSET:WS_STATUS_OFFSET + 4].cpu().numpy().view("<u4")[0])


def _dev(t, dtype, name):
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def characterize(text, offsets, counts=None, ws=None, validate=False):
    """Word counts (str.split() semantics) of the prompts text[offsets[i]:offsets[i+1]]."""
    _dev(text, torch.uint8, "text")
    _dev(offsets, torch.int64, "offsets")
    n = offsets.numel() - 1
    if counts is None:
        counts = torch.empty(max(n, 0), dtype=torch.int32, device=offsets.device)
    _dev(counts, torch.int32, "counts")
    if ws is None:
        ws = workspace(OP_CHARACTERIZE, n, 0, offsets.device)
    _check(lib.ds_characterize(_ptr(text) if text.numel() else None, text.numel(), _ptr(offsets), n,
                               _ptr(counts), _ptr(ws), ws.numel(), _flags(validate), _stream()))
    return counts


def calibrate(group, est, observed, alpha, state, trace=True, ws=None, validate=False,
              trace_before=None, no_wait=False):
    """EMA calibration factors (Eq. 5/6). Updates ``state`` in place.

    Returns (state, trace or None), and the factors before each event as a
    third item when ``trace_before`` is True or a tensor."""
    _dev(group, torch.int32, "group")
    _dev(est, torch.float64, "est")
    _dev(observed, torch.int32, "observed")
    _dev(state, torch.float64, "state")
    n = group.numel()

    def out_arg(x, name):
        if x is True:
            return torch.empty(n, dtype=torch.float64, device=group.device)
        if x is None or x is False:
            return None
        return _dev(x, torch.float64, name)

    tr = out_arg(trace, "trace")
    tb = out_arg(trace_before, "trace_before")
    if ws is None:
        ws = workspace(OP_CALIBRATE, n, state.numel(), group.device)
    _check(lib.ds_calibrate_ex(_ptr(group), _ptr(est), _ptr(observed), n, float(alpha),
                               state.numel(), _ptr(state), _ptr(tr), _ptr(tb), _ptr(ws), ws.numel(),
                               _flags(validate, no_wait), _stream()))
    if trace_before is None or trace_before is False:
        return state, tr
    return state, tr, tb


def error_stats(est, observed, factor=None, group=None, n_groups=0, out=None, ws=None,
                validate=False):
    """MAE, RMSE and mean bias of est * factor against observed, per group and
    overall (tab:four_mode_token_error). Returns a (n_groups + 1, 4) float64
    tensor: count, MAE, RMSE, mean bias; the last row covers all events."""
    _dev(est, torch.float64, "est")
    _dev(observed, torch.int32, "observed")
    if factor is not None:
        _dev(factor, torch.float64, "factor")
    if group is not None:
        _dev(group, torch.int32, "group")
    n = est.numel()
    dev = est.device
    if out is None:
        out = torch.empty((n_groups + 1, 4), dtype=torch.float64, device=dev)
    _dev(out, torch.float64, "out")
    if ws is None:
        ws = workspace(OP_ERROR_STATS, n, n_groups, dev)
    _check(lib.ds_error_stats(n, _ptr(est), _ptr(factor), _ptr(observed), _ptr(group), int(n_groups),
                              _ptr(out), _ptr(ws), ws.numel(), _flags(validate), _stream()))
    return out


READ_BW_WORDS = 32768


def read_bandwidth(buf, out=None):
    """The read side of characterize alone over a contiguous device tensor
    (its size a multiple of 16 bytes). Returns an int32 tensor of
    READ_BW_WORDS words whose XOR is the XOR of the buffer's 32-bit words."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    if out is None:
        out = torch.empty(READ_BW_WORDS, dtype=torch.int32, device=buf.device)
    _dev(out, torch.int32, "out")
    nbytes = buf.numel() * buf.element_size()
    _check(lib.ds_read_bandwidth(_ptr(buf) if nbytes else None, nbytes, _ptr(out), _stream()))
    return out


def class_histogram(category, job_class, n_cat, out=None, ws=None, validate=False):
    """Requests per (category, runtime class): a (n_cat, 3) int32 tensor."""
    _dev(category, torch.uint8, "category")
    _dev(job_class, torch.uint8, "job_class")
    n = category.numel()
    dev = category.device
    if out is None:
        out = torch.empty((n_cat, 3), dtype=torch.int32, device=dev)
    _dev(out, torch.int32, "out")
    if ws is None and validate:
        ws = workspace(OP_CLASS_HIST, n, 0, dev)
    _check(lib.ds_class_histogram(n, _ptr(category), int(n_cat), _ptr(job_class), _ptr(out),
                                  _ptr(ws), ws.numel() if ws is not None else 0, _flags(validate),
                                  _stream()))
    return out


def score(counts, category, tenant, group, t_base, s_tenant, state, f_ref=1024.0,
          short_max=128.0, medium_max=512.0, want_est_base=True, out=None, ws=None,
          validate=False):
    """Budget estimate (Eq. 1/2) and class (Eq. 4). Returns (est_base, est, budget, class).

    ``group`` None: ``state`` holds one factor per request (as-of scoring)."""
    _dev(counts, torch.int32, "counts")
    _dev(category, torch.uint8, "category")
    _dev(tenant, torch.int32, "tenant")
    if group is not None:
        _dev(group, torch.int32, "group")
    _dev(t_base, torch.float64, "t_base")
    _dev(s_tenant, torch.float64, "s_tenant")
    _dev(state, torch.float64, "state")
    n = counts.numel()
    dev = counts.device
    if out is None:
        est_base = torch.empty(n, dtype=torch.float64, device=dev) if want_est_base else None
        est = torch.empty(n, dtype=torch.float64, device=dev)
        budget = torch.empty(n, dtype=torch.float64, device=dev)
        cls = torch.empty(n, dtype=torch.uint8, device=dev)
    else:
        est_base, est, budget, cls = out
    if ws is None and validate:
        ws = workspace(OP_SCORE, n, 0, dev)
    p = ScoreParams(float(f_ref), float(short_max), float(medium_max))
    _check(lib.ds_score(n, _ptr(counts), _ptr(category), _ptr(tenant), _ptr(group), _ptr(t_base),
                        t_base.numel(), _ptr(s_tenant), s_tenant.numel(), _ptr(state), state.numel(),
                        ctypes.byref(p), _ptr(est_base), _ptr(est), _ptr(budget), _ptr(cls),
                        _ptr(ws), ws.numel() if ws is not None else 0, _flags(validate), _stream()))
    return est_base, est, budget, cls


def characterize_score(text, offsets, category, tenant, group, t_base, s_tenant, state,
                       f_ref=1024.0, short_max=128.0, medium_max=512.0, want_est_base=True,
                       counts=None, out=None, ws=None, validate=False):
    """``characterize`` then ``score`` on its counts, in one pass (the same
    results). Returns (counts, (est_base, est, budget, class))."""
    _dev(text, torch.uint8, "text")
    _dev(offsets, torch.int64, "offsets")
    for t, dt, name in ((category, torch.uint8, "category"), (tenant, torch.int32, "tenant"),
                        (group, torch.int32, "group"), (t_base, torch.float64, "t_base"),
                        (s_tenant, torch.float64, "s_tenant"), (state, torch.float64, "state")):
        if t is not None or name != "group":
            _dev(t, dt, name)
    n = offsets.numel() - 1
    dev = offsets.device
    if counts is None:
        counts = torch.empty(max(n, 0), dtype=torch.int32, device=dev)
    _dev(counts, torch.int32, "counts")
    if out is None:
        m = max(n, 0)
        est_base = torch.empty(m, dtype=torch.float64, device=dev) if want_est_base else None
        out = (est_base, torch.empty(m, dtype=torch.float64, device=dev),
               torch.empty(m, dtype=torch.float64, device=dev), torch.empty(m, dtype=torch.uint8, device=dev))
    est_base, est, budget, cls = out
    if ws is None:
        ws = workspace(OP_CHARACTERIZE, n, 0, dev)
    p = ScoreParams(float(f_ref), float(short_max), float(medium_max))
    _check(lib.ds_characterize_score(_ptr(text) if text.numel() else None, text.numel(), _ptr(offsets), n,
                                     _ptr(counts), _ptr(category), _ptr(tenant), _ptr(group), _ptr(t_base),
                                     t_base.numel(), _ptr(s_tenant), s_tenant.numel(), _ptr(state),
                                     state.numel(), ctypes.byref(p), _ptr(est_base), _ptr(est), _ptr(budget),
                                     _ptr(cls), _ptr(ws), ws.numel(), _flags(validate), _stream()))
    return counts, out


NOALLOC_MAX_PROMPTS = 1 << 20


def characterize_score_noalloc(text, offsets, category, tenant, group, t_base, s_tenant, state,
                               f_ref=1024.0, short_max=128.0, medium_max=512.0, counts=None,
                               out=None):
    """``characterize_score`` through ds_characterize_score_noalloc: no
    workspace (the library's static scratch array). ``counts`` and ``out``
    (est_base or None, est, budget, class) are the caller's tensors; the
    call itself allocates nothing. Returns (counts, out)."""
    _dev(text, torch.uint8, "text")
    _dev(offsets, torch.int64, "offsets")
    for t, dt, name in ((category, torch.uint8, "category"), (tenant, torch.int32, "tenant"),
                        (group, torch.int32, "group"), (t_base, torch.float64, "t_base"),
                        (s_tenant, torch.float64, "s_tenant"), (state, torch.float64, "state"),
                        (counts, torch.int32, "counts")):
        _dev(t, dt, name)
    n = offsets.numel() - 1
    est_base, est, budget, cls = out
    p = ScoreParams(float(f_ref), float(short_max), float(medium_max))
    _check(lib.ds_characterize_score_noalloc(
        _ptr(text) if text.numel() else None, text.numel(), _ptr(offsets), n, _ptr(counts),
        _ptr(category), _ptr(tenant), _ptr(group), _ptr(t_base), t_base.numel(), _ptr(s_tenant),
        s_tenant.numel(), _ptr(state), state.numel(), ctypes.byref(p), _ptr(est_base), _ptr(est),
        _ptr(budget), _ptr(cls), 0, _stream()))
    return counts, out


def order_params(n_tiers=3, weights=(4, 2, 1), tier_priority=(0.0, 1.0, 2.0), aging_rate=0.01,
                 t_now=0.0, aging_floor=0.0, weighted_mode=WRR_BLOCKED):
    """ds_order_params. weighted_mode: WRR_BLOCKED, WRR_SMOOTH or WRR_STRIDE
    (or their names "blocked", "smooth", "stride")."""
    if isinstance(weighted_mode, str):
        weighted_mode = {"blocked": WRR_BLOCKED, "smooth": WRR_SMOOTH, "stride": WRR_STRIDE}[weighted_mode]
    p = OrderParams()
    p.n_tiers = int(n_tiers)
    for q in range(MAX_TIERS):
        p.weight[q] = int(weights[q]) if q < len(weights) else 1
        p.tier_priority[q] = float(tier_priority[q]) if q < len(tier_priority) else 0.0
    p.aging_rate = float(aging_rate)
    p.t_now = float(t_now)
    p.aging_floor = float(aging_floor)
    p.weighted_mode = int(weighted_mode)
    return p


def order(policy, tier, arrival, budget=None, fifo=None, params=None, perm=None, key=False,
          ws=None, validate=False, serial_sort=False, no_wait=False, **kw):
    """Dispatch permutation of one policy. Returns (perm, key or None).

    ``serial_sort`` sets DS_SERIAL_SORT (the single-workgroup sort; a
    diagnostic)."""
    if isinstance(policy, str):
        policy = POLICIES[policy]
    _dev(tier, torch.uint8, "tier")
    _dev(arrival, torch.float64, "arrival")
    if budget is not None:
        _dev(budget, torch.float64, "budget")
    if fifo is not None:
        _dev(fifo, torch.int32, "fifo")
    n = tier.numel()
    dev = tier.device
    if params is None:
        params = order_params(**kw)
    if perm is None:
        perm = torch.empty(n, dtype=torch.int32, device=dev)
    k = None
    if key is True:
        k = torch.empty(n, dtype=torch.float64, device=dev)
    elif key is not False and key is not None:
        k = _dev(key, torch.float64, "key")
    if ws is None:
        ws = workspace(OP_ORDER, n, 0, dev)
    flags = _flags(validate, no_wait) | (DS_SERIAL_SORT if serial_sort else 0)
    _check(lib.ds_order(int(policy), n, _ptr(tier), _ptr(arrival), _ptr(budget), _ptr(fifo),
                        ctypes.byref(params), _ptr(perm), _ptr(k), _ptr(ws), ws.numel(),
                        flags, _stream()))
    return perm, k


def order_multi(policies, tier, arrival, budget=None, fifo=None, params=None, perms=None,
                keys=False, ws=None, validate=False, serial_sort=False, no_wait=False, **kw):
    """Dispatch permutations of several policies in one call (FIFO computed
    once, the policy sorts batched). Returns ({policy: perm}, {policy: key})."""
    pols = [POLICIES[p] if isinstance(p, str) else int(p) for p in policies]
    mask = 0
    for p in pols:
        mask |= 1 << p
    _dev(tier, torch.uint8, "tier")
    _dev(arrival, torch.float64, "arrival")
    if budget is not None:
        _dev(budget, torch.float64, "budget")
    if fifo is not None:
        _dev(fifo, torch.int32, "fifo")
    n = tier.numel()
    dev = tier.device
    if params is None:
        params = order_params(**kw)
    out_p, out_k = {}, {}
    pp = (ctypes.c_void_p * 5)()
    kk = (ctypes.c_void_p * 5)()
    for p in pols:
        t = perms[p] if perms is not None and p in perms else torch.empty(n, dtype=torch.int32, device=dev)
        _dev(t, torch.int32, "perm")
        out_p[p] = t
        pp[p] = t.data_ptr()
        if keys:
            k = torch.empty(n, dtype=torch.float64, device=dev)
            out_k[p] = k
            kk[p] = k.data_ptr()
    if ws is None:
        ws = workspace(OP_ORDER_MULTI, n, 0, dev)
    flags = _flags(validate, no_wait) | (DS_SERIAL_SORT if serial_sort else 0)
    _check(lib.ds_order_multi(mask, n, _ptr(tier), _ptr(arrival), _ptr(budget), _ptr(fifo),
                              ctypes.byref(params), pp, kk if keys else None, _ptr(ws), ws.numel(),
                              flags, _stream()))
    return out_p, out_k


def sim_params(policy, batch=32, alpha=0.1, f_ref=1024.0, **order_kw):
    """ds_sim_params for ``simulate`` (order_kw as ``order_params``)."""
    if isinstance(policy, str):
        policy = POLICIES[policy]
    p = SimParams()
    p.policy = int(policy)
    p.batch = int(batch)
    p.alpha = float(alpha)
    p.score = ScoreParams(float(f_ref), 128.0, 512.0)
    p.order = order_params(**order_kw)
    return p


def simulate(arrival, tier, counts, category, tenant, group, observed, t_base, s_tenant, state,
             tick_t, params, out=None, ws=None, validate=False):
    """Dispatch ticks of the online loop; ``state`` is updated in place.

    Returns (seq, tick_of, n_dispatched): device tensors (int32 x2, and one
    int32 element) without a host synchronisation.
    """
    _dev(arrival, torch.float64, "arrival")
    _dev(tier, torch.uint8, "tier")
    _dev(counts, torch.int32, "counts")
    _dev(category, torch.uint8, "category")
    _dev(tenant, torch.int32, "tenant")
    _dev(group, torch.int32, "group")
    _dev(observed, torch.int32, "observed")
    _dev(t_base, torch.float64, "t_base")
    _dev(s_tenant, torch.float64, "s_tenant")
    _dev(state, torch.float64, "state")
    _dev(tick_t, torch.float64, "tick_t")
    n = arrival.numel()
    dev = arrival.device
    if out is None:
        seq = torch.empty(n, dtype=torch.int32, device=dev)
        tick_of = torch.empty(n, dtype=torch.int32, device=dev)
        nd = torch.empty(1, dtype=torch.int32, device=dev)
    else:
        seq, tick_of, nd = out
    if ws is None:
        ws = workspace(OP_SIMULATE, n, 0, dev)
    _check(lib.ds_simulate(n, _ptr(arrival), _ptr(tier), _ptr(counts), _ptr(category),
                           _ptr(tenant), _ptr(group), _ptr(observed), _ptr(t_base),
                           t_base.numel(), _ptr(s_tenant), s_tenant.numel(), state.numel(),
                           _ptr(tick_t), tick_t.numel(), ctypes.byref(params), _ptr(state),
                           _ptr(seq), _ptr(tick_of), _ptr(nd), _ptr(ws), ws.numel(),
                           _flags(validate), _stream()))
    return seq, tick_of, nd


def simulate_multi(arrival, tier, counts, category, tenant, group, observed, t_base, s_tenant,
                   states, tick_t, params, ws=None, validate=False):
    """Several dispatch-tick loops in one launch (ds_simulate_multi): run r
    uses params[r] and updates states[r] in place. Returns a list of
    (seq, tick_of) per run and the n_dispatched tensor (one int32 per run)."""
    for t, dt, name in ((arrival, torch.float64, "arrival"), (tier, torch.uint8, "tier"),
                        (counts, torch.int32, "counts"), (category, torch.uint8, "category"),
                        (tenant, torch.int32, "tenant"), (group, torch.int32, "group"),
                        (observed, torch.int32, "observed"), (t_base, torch.float64, "t_base"),
                        (s_tenant, torch.float64, "s_tenant"), (tick_t, torch.float64, "tick_t")):
        _dev(t, dt, name)
    R = len(params)
    if R != len(states):
        raise ValueError("one state per run")
    for st in states:
        _dev(st, torch.float64, "state")
    n = arrival.numel()
    dev = arrival.device
    outs = [(torch.empty(n, dtype=torch.int32, device=dev), torch.empty(n, dtype=torch.int32, device=dev))
            for _ in range(R)]
    nd = torch.empty(R, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(OP_SIMULATE_MULTI, n, R, dev)
    P = ctypes.c_void_p
    pa = (SimParams * R)(*params)
    st_p = (P * R)(*[st.data_ptr() for st in states])
    sq_p = (P * R)(*[o[0].data_ptr() for o in outs])
    tk_p = (P * R)(*[o[1].data_ptr() for o in outs])
    n_groups = states[0].numel() if states else 1
    _check(lib.ds_simulate_multi(R, n, _ptr(arrival), _ptr(tier), _ptr(counts), _ptr(category),
                                 _ptr(tenant), _ptr(group), _ptr(observed), _ptr(t_base),
                                 t_base.numel(), _ptr(s_tenant), s_tenant.numel(), n_groups,
                                 _ptr(tick_t), tick_t.numel(), pa, st_p, sq_p, tk_p, _ptr(nd),
                                 _ptr(ws), ws.numel(), _flags(validate), _stream()))
    return outs, nd
