"""Plain single-threaded CPU oracle for the DriftSched admission hot path.

TEST INFRASTRUCTURE. Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. The product path
(the HIP library under ``paper_2606_02982_amd``) never imports it and shares
no code with it.

The arithmetic lives in ``driftsched_ref.c`` (plain loops, fp64, built with
``-ffp-contract=off``); this module only builds that file and marshals numpy
arrays to it. Each wrapper names the passage of the paper it follows; the C
file carries the full statement.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "driftsched_ref.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

FIFO, PRIORITY, WEIGHTED, SJF, AGING = 0, 1, 2, 3, 4
WEIGHTED_SMOOTH = 5   # the smooth weighted round robin reading of Weighted
WEIGHTED_STRIDE = 6   # the stride scheduling reading of Weighted


def build(force=True):
    """Compile the oracle with gcc (plain C11, no fused multiply-add)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=gnu11", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"]
    subprocess.check_call(cmd)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    u32, u64, f64, i32 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_double, ctypes.c_int
    lib.dsref_is_space.argtypes = [u32]
    lib.dsref_is_space.restype = i32
    lib.dsref_count_words.argtypes = [P, u64]
    lib.dsref_count_words.restype = u32
    lib.dsref_characterize.argtypes = [P, u64, P, u64, P]
    lib.dsref_characterize.restype = i32
    lib.dsref_calibrate.argtypes = [P, P, P, u64, f64, u32, P, P]
    lib.dsref_calibrate.restype = i32
    lib.dsref_calibrate_ex.argtypes = [P, P, P, u64, f64, u32, P, P, P]
    lib.dsref_calibrate_ex.restype = i32
    lib.dsref_error_stats.argtypes = [u64, P, P, P, P, u32, P]
    lib.dsref_error_stats.restype = i32
    lib.dsref_class_histogram.argtypes = [u64, P, u32, P, P]
    lib.dsref_class_histogram.restype = i32
    lib.dsref_score.argtypes = [u64, P, P, P, P, P, u32, P, u32, P, u32,
                                f64, f64, f64, P, P, P, P]
    lib.dsref_score.restype = i32
    lib.dsref_order.argtypes = [i32, u32, P, P, P, u32, P, P, f64, f64, f64, P, P]
    lib.dsref_order.restype = i32
    lib.dsref_simulate.argtypes = [i32, u32, P, P, P, P, P, P, P, P, u32, P, u32, u32,
                                   f64, f64, f64, u32, P, P, f64, f64, f64, u32, P, u32, P,
                                   P, P, P]
    lib.dsref_simulate.restype = i32
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def is_space(cp):
    """Membership of code point cp in str.split()'s separator set."""
    return bool(_load().dsref_is_space(int(cp)))


def count_words(b):
    """len(b.decode('utf-8', 'surrogateescape').split()) for one prompt (bytes)."""
    arr = np.frombuffer(bytes(b), dtype=np.uint8)
    return int(_load().dsref_count_words(_ptr(arr) if len(arr) else None, len(arr)))


def characterize(text, offsets):
    """Stage 1: per-prompt whitespace-proxy counts (Sec. Workload Characterization)."""
    text = _c(text, np.uint8)
    offsets = _c(offsets, np.uint64)
    n = len(offsets) - 1
    counts = np.zeros(max(n, 0), dtype=np.uint32)
    rc = _load().dsref_characterize(_ptr(text), len(text), _ptr(offsets), n, _ptr(counts))
    if rc != 0:
        raise ValueError("oracle characterize: offsets not nondecreasing or beyond the text")
    return counts


def calibrate(group, est, obs, alpha, state, with_trace=True, with_before=False):
    """Stage 2: EMA of Eq. (5) over ratios of Eq. (6), events in completion order.

    Returns (state_out, trace or None), and trace_before (the factor of each
    event's group just before it) as a third item when ``with_before``;
    ``state`` is not modified.
    """
    group = _c(group, np.uint32)
    est = _c(est, np.float64)
    obs = _c(obs, np.uint32)
    st = np.array(state, dtype=np.float64, copy=True)
    n = len(group)
    trace = np.zeros(n, dtype=np.float64) if with_trace else None
    before = np.zeros(n, dtype=np.float64) if with_before else None
    rc = _load().dsref_calibrate_ex(_ptr(group), _ptr(est), _ptr(obs), n, float(alpha),
                                    len(st), _ptr(st), _ptr(trace), _ptr(before))
    if rc != 0:
        raise ValueError("oracle calibrate: group index out of range")
    return (st, trace, before) if with_before else (st, trace)


def error_stats(est, obs, factor=None, group=None, n_groups=0):
    """Estimation error per group and overall: array (n_groups + 1, 4) of
    count, MAE, RMSE, mean bias (tab:four_mode_token_error)."""
    est = _c(est, np.float64)
    obs = _c(obs, np.uint32)
    fac = None if factor is None else _c(factor, np.float64)
    grp = None if group is None else _c(group, np.uint32)
    out = np.zeros(4 * (n_groups + 1), dtype=np.float64)
    rc = _load().dsref_error_stats(len(est), _ptr(est), _ptr(fac), _ptr(obs), _ptr(grp),
                                   int(n_groups), _ptr(out))
    if rc != 0:
        raise ValueError("oracle error_stats: group index out of range")
    return out.reshape(n_groups + 1, 4)


def class_histogram(category, job_class, n_cat):
    """Runtime classes per category: array (n_cat, 3) of counts."""
    category = _c(category, np.uint8)
    job_class = _c(job_class, np.uint8)
    out = np.zeros(3 * n_cat, dtype=np.uint32)
    rc = _load().dsref_class_histogram(len(category), _ptr(category), int(n_cat),
                                       _ptr(job_class), _ptr(out))
    if rc != 0:
        raise ValueError("oracle class_histogram: category or class out of range")
    return out.reshape(n_cat, 3)


def score(counts, category, tenant, group, t_base, s_tenant, state,
          f_ref=1024.0, short_max=128.0, medium_max=512.0):
    """Stage 3: Eq. (1)/(2) in Alg. 1's order and the classes of Eq. (4).

    ``group`` None: ``state`` holds one factor per request (as-of scoring).
    Returns (est_base, est, budget, job_class).
    """
    counts = _c(counts, np.uint32)
    category = _c(category, np.uint8)
    tenant = _c(tenant, np.uint32)
    group = None if group is None else _c(group, np.uint32)
    t_base = _c(t_base, np.float64)
    s_tenant = _c(s_tenant, np.float64)
    state = _c(state, np.float64)
    n = len(counts)
    est_base = np.zeros(n, np.float64)
    est = np.zeros(n, np.float64)
    budget = np.zeros(n, np.float64)
    cls = np.zeros(n, np.uint8)
    rc = _load().dsref_score(n, _ptr(counts), _ptr(category), _ptr(tenant), _ptr(group),
                             _ptr(t_base), len(t_base), _ptr(s_tenant), len(s_tenant),
                             _ptr(state), len(state), float(f_ref), float(short_max),
                             float(medium_max), _ptr(est_base), _ptr(est), _ptr(budget),
                             _ptr(cls))
    if rc != 0:
        raise ValueError("oracle score: index out of range")
    return est_base, est, budget, cls


def order(policy, tier, arrival, budget=None, weights=(4, 2, 1),
          tier_priority=(0.0, 1.0, 2.0), aging_rate=0.01, t_now=0.0, aging_floor=0.0):
    """Stage 4: dispatch permutation of one policy and each request's key."""
    tier = _c(tier, np.uint8)
    arrival = _c(arrival, np.float64)
    n = len(tier)
    b = _c(budget, np.float64) if budget is not None else np.zeros(n, np.float64)
    w = _c(weights, np.uint32)
    tp = _c(tier_priority, np.float64)
    if len(w) != len(tp):
        raise ValueError("weights and tier_priority must have one entry per tier")
    perm = np.zeros(n, np.uint32)
    key = np.zeros(n, np.float64)
    rc = _load().dsref_order(int(policy), n, _ptr(tier), _ptr(arrival), _ptr(b), len(w),
                             _ptr(w), _ptr(tp), float(aging_rate), float(t_now),
                             float(aging_floor), _ptr(perm), _ptr(key))
    if rc != 0:
        raise ValueError("oracle order: bad tier, weight or policy")
    return perm, key


def simulate(policy, arrival, tier, counts, category, tenant, group, observed, t_base,
             s_tenant, state, tick_t, batch=32, alpha=0.1, weights=(4, 2, 1),
             tier_priority=(0.0, 1.0, 2.0), aging_rate=0.01, aging_floor=0.0,
             f_ref=1024.0, short_max=128.0, medium_max=512.0):
    """Dispatch ticks of the online loop: order the pending set, dispatch a
    batch, fold its completions into the factors (dsref_simulate).

    Returns (seq[:n_dispatched], tick_of, state after the last tick).
    """
    arrival = _c(arrival, np.float64)
    tier = _c(tier, np.uint8)
    counts = _c(counts, np.uint32)
    category = _c(category, np.uint8)
    tenant = _c(tenant, np.uint32)
    group = _c(group, np.uint32)
    observed = _c(observed, np.uint32)
    t_base = _c(t_base, np.float64)
    s_tenant = _c(s_tenant, np.float64)
    st = np.array(state, dtype=np.float64)
    tick_t = _c(tick_t, np.float64)
    w = _c(weights, np.uint32)
    tp = _c(tier_priority, np.float64)
    if len(w) != len(tp):
        raise ValueError("weights and tier_priority must have one entry per tier")
    n = len(arrival)
    seq = np.zeros(n, np.uint32)
    tick_of = np.zeros(n, np.int32)
    nd = ctypes.c_uint32(0)
    rc = _load().dsref_simulate(int(policy), n, _ptr(arrival), _ptr(tier), _ptr(counts),
                                _ptr(category), _ptr(tenant), _ptr(group), _ptr(observed),
                                _ptr(t_base), len(t_base), _ptr(s_tenant), len(s_tenant),
                                len(st), float(f_ref), float(short_max), float(medium_max),
                                len(w), _ptr(w), _ptr(tp), float(aging_rate),
                                float(aging_floor), float(alpha), int(batch), _ptr(tick_t),
                                len(tick_t), _ptr(st), _ptr(seq), _ptr(tick_of),
                                ctypes.byref(nd))
    if rc != 0:
        raise ValueError("oracle simulate: bad index, weight, policy or batch")
    return seq[:nd.value], tick_of, st
