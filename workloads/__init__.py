"""Seeded synthetic workloads for the DriftSched admission hot path.

A module of its own, outside the HIP package and outside the oracle: it only
makes inputs, and both sides receive the arrays it returns unchanged. It holds
none of the four stages' arithmetic: no word counting, no budget estimate
(the product of the baseline, the tenant scaling and the prompt-complexity
factor), no calibration update, no class, no policy key or ordering.

The workloads define each request's observed output length as its B-free
admission estimate times a log-normal drift ratio. That estimate is the score
stage's output, so this module draws the ratios only; ``complete()`` turns an
estimate computed elsewhere (by the CPU oracle in the tests, by the library's
own score call during benchmark set-up) into the completion events.

The paper's own prompt corpus (about 1,180 prompts in four semantic
categories, three tenant tiers) is not available; these generators stand in
for it with the shapes the workloads below state: packed UTF-8 prompt
buffers of random lowercase words separated by runs of space/tab/newline,
Poisson arrivals, tenants spread uniformly over the three tiers, four
semantic categories, and log-normal ratios between observed and estimated
output length. No item of any corpus is reproduced.

Per-request arrays come from numpy's PCG64 generator seeded per workload; the
prompt text comes from a counter-based SplitMix64 stream per prompt (see
synth_text.c), so that it does not depend on how the other arrays are drawn.
"""
import ctypes
from dataclasses import dataclass
import os
import subprocess

import numpy as np

# Per-category baseline output estimates T_base for short_qa, summary,
# technical, report. The paper names the symbol but prints no values; these
# are this implementation's inputs (dyadic, so hand cases stay exact).
T_BASE = (32.0, 128.0, 256.0, 512.0)
# Tenant safety scaling S per tier (Premium, Standard, Batch); inputs likewise.
S_TIER = (1.25, 1.125, 1.0)
# Reference prompt length of the prompt-complexity factor F = 1 + n / F_REF.
F_REF = 1024.0
# Tier priorities: Premium first.
TIER_PRIORITY = (0.0, 1.0, 2.0)
N_TIERS = 3


# Two- and three-byte letters used where a workload asks for non-ASCII text.
# Several share a lead byte, or lead and second byte, with multi-byte
# whitespace (C2 85, C2 A0, E2 80 80..8A, E3 80 80, E1 9A 80) without being
# whitespace themselves.
NONASCII_LETTERS = ("\u00c5", "\u00e0", "\u00b5", "\u0420", "\u00a9", "\u03bb",
                    "\u2c65", "\u3042", "\u4e00", "\u2010", "\u1e00", "\u3007")


@dataclass(frozen=True)
class Workload:
    name: str
    n: int                       # requests in the batch (or completion events)
    words: tuple                 # (lo, hi) words per prompt, uniform
    tenants: int
    ratio_mu: float = 0.25       # ln(observed / estimate) ~ N(mu, sigma^2)
    ratio_sigma: float = 0.3
    tenant_offset_sd: float = 0.0
    nonascii_p: float = 0.0      # probability that a letter is non-ASCII
    alphas: tuple = (0.1,)
    seed: int = 0
    rate: float = 5000.0         # Poisson arrivals per second
    aging_rate: float = 0.01     # priority units per second of waiting
    weights: tuple = (4, 2, 1)
    has_text: bool = True
    drift_means: tuple = ()      # piecewise ratio means (event-indexed)
    drift_steps: tuple = ()      # event indices where the mean steps
    ticks: int = 0               # aging re-sort ticks
    policies: tuple = ("fifo", "priority", "weighted", "sjf", "aging")
    note: str = ""


WORKLOADS = {
    "batch4k": Workload(
        "batch4k", 4096, (16, 512), 8, 0.25, 0.3, seed=0,
        note="4,096 requests, 8 tenants, 16-512 words, weights 4/2/1, all five policies"),
    "batch64k": Workload(
        "batch64k", 65536, (32, 2048), 64, 0.3, 0.4, tenant_offset_sd=0.1, seed=1,
        note="65,536 requests, 64 tenants, 32-2,048 words, per-tenant ratio offset"),
    "chat1m": Workload(
        "chat1m", 1048576, (8, 256), 1024, 0.25, 0.3, seed=2,
        note="1,048,576 short chat requests, 1,024 tenants, 8-256 words"),
    "long16k": Workload(
        "long16k", 16384, (8192, 32768), 16, 0.25, 0.3, nonascii_p=0.02696, seed=3,
        note="16,384 long-context prompts of 8,192-32,768 words, ~5% non-ASCII bytes"),
    "drift4m": Workload(
        "drift4m", 4194304, (8, 256), 4096, 0.0, 0.3, alphas=(0.05, 0.2), seed=4,
        has_text=False, drift_means=(0.8, 1.4, 1.0), drift_steps=(1 << 20, 3 << 20),
        ticks=64, policies=("aging",),
        note="4,194,304 completion events, 4,096 tenants, ratio mean 0.8->1.4->1.0"),
}


class Batch(dict):
    """A dict of arrays with attribute access."""
    __getattr__ = dict.__getitem__


def _assert_letters_not_space():
    for ch in NONASCII_LETTERS:
        if ch.isspace():
            raise AssertionError("non-ASCII letter pool contains whitespace: %r" % ch)


_HERE = os.path.dirname(os.path.abspath(__file__))
_TEXT_SRC = os.path.join(_HERE, "synth_text.c")
_TEXT_LIB = os.path.join(_HERE, "libsynth_text.so")
_text_lib = None


def build_text_lib():
    """Compile the text synthesiser (plain C, OpenMP over prompts)."""
    tmp = _TEXT_LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-std=gnu11", "-O2", "-fopenmp", "-fPIC", "-shared",
                           "-Wall", "-o", tmp, _TEXT_SRC])
    os.replace(tmp, _TEXT_LIB)
    return _TEXT_LIB


def _load_text_lib():
    global _text_lib
    if _text_lib is None:
        if not os.path.exists(_TEXT_LIB):
            build_text_lib()
        lib = ctypes.CDLL(_TEXT_LIB)
        P = ctypes.c_void_p
        lib.synth_text.argtypes = [ctypes.c_uint64, P, ctypes.c_uint64, ctypes.c_double, P, P, P]
        lib.synth_text.restype = ctypes.c_int64
        _text_lib = lib
    return _text_lib


def make_text(words, seed, nonascii_p=0.0):
    """Packed prompt buffer for prompts with the given word counts (>= 1).

    Returns (text uint8[B], offsets uint64[n+1]); prompt i is
    text[offsets[i]:offsets[i+1]].
    """
    _assert_letters_not_space()
    lib = _load_text_lib()
    words = np.ascontiguousarray(words, dtype=np.uint32)
    n = len(words)
    lengths = np.zeros(n, dtype=np.uint64)
    wp = words.ctypes.data_as(ctypes.c_void_p)
    total = lib.synth_text(seed, wp, n, float(nonascii_p), None, None,
                           lengths.ctypes.data_as(ctypes.c_void_p))
    offsets = np.zeros(n + 1, dtype=np.uint64)
    np.cumsum(lengths, out=offsets[1:])
    text = np.empty(int(total), dtype=np.uint8)
    if total:
        lib.synth_text(seed, wp, n, float(nonascii_p), text.ctypes.data_as(ctypes.c_void_p),
                       offsets.ctypes.data_as(ctypes.c_void_p), None)
    return text, offsets


def generate(wl, n=None, with_text=True):
    """Arrays for workload ``wl`` (a Workload or its name).

    ``n`` overrides the request count (for reduced test cases) keeping every
    other parameter. Arrays are in batch order: the batch lists the requests
    in a seeded random permutation of arrival order, so that FIFO is a real
    sort. Completion events are the same requests in arrival order:
    ``ev_req[e]`` is the batch index of event e's request, ``ev_group[e]`` its
    calibration group and ``ev_ratio[e]`` the drift ratio of its observed
    length. The events' estimates and observed lengths are added by
    ``complete()``.
    """
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    n = wl.n if n is None else int(n)
    rng = np.random.default_rng(wl.seed)
    lo, hi = wl.words
    words = rng.integers(lo, hi + 1, n, dtype=np.int64)
    tenant = rng.integers(0, wl.tenants, n, dtype=np.int64)
    category = rng.integers(0, len(T_BASE), n, dtype=np.int64)
    gaps = rng.exponential(1.0 / wl.rate, n)
    arrival_sorted = np.cumsum(gaps)
    if wl.has_text:
        rank = rng.permutation(n)          # batch position j holds arrival rank rank[j]
    else:
        rank = np.arange(n)                # stored in arrival order
    if wl.drift_means:
        e = np.arange(n)
        seg = np.searchsorted(np.asarray(wl.drift_steps), e, side="right")
        m = np.asarray(wl.drift_means)[seg]
        mu = np.log(m) - 0.5 * wl.ratio_sigma ** 2
        ratio_by_rank = np.exp(rng.normal(mu, wl.ratio_sigma))
    else:
        offs = (rng.normal(0.0, wl.tenant_offset_sd, wl.tenants)
                if wl.tenant_offset_sd > 0 else np.zeros(wl.tenants))
        ratio_by_rank = None
        ln_ratio = rng.normal(wl.ratio_mu, wl.ratio_sigma, n)
    tier = (tenant % N_TIERS).astype(np.uint8)
    s_tenant = np.asarray(S_TIER, dtype=np.float64)[np.arange(wl.tenants) % N_TIERS]
    t_base = np.asarray(T_BASE, dtype=np.float64)

    out = Batch()
    out["workload"] = wl
    out["n"] = n
    out["words"] = words.astype(np.uint32)
    out["tenant"] = tenant.astype(np.uint32)
    out["group"] = tenant.astype(np.uint32)
    out["category"] = category.astype(np.uint8)
    out["tier"] = tier
    out["arrival"] = arrival_sorted[rank]
    out["t_base"] = t_base
    out["s_tenant"] = s_tenant
    out["f_ref"] = F_REF
    out["n_groups"] = wl.tenants
    out["weights"] = np.asarray(wl.weights, dtype=np.uint32)
    out["tier_priority"] = np.asarray(TIER_PRIORITY, dtype=np.float64)
    out["aging_rate"] = wl.aging_rate
    out["aging_floor"] = 0.0
    out["t_now"] = float(arrival_sorted[-1]) if n else 0.0
    out["alphas"] = wl.alphas

    # completion events: the same requests in arrival order
    by_arrival = np.empty(n, dtype=np.int64)
    by_arrival[rank] = np.arange(n)
    if ratio_by_rank is None:
        ratio = np.exp(ln_ratio + offs[tenant])          # batch order
        ratio_ev = ratio[by_arrival]
    else:
        ratio_ev = ratio_by_rank
    out["ev_req"] = by_arrival
    out["ev_group"] = tenant[by_arrival].astype(np.uint32)
    out["ev_ratio"] = ratio_ev

    if wl.has_text and with_text:
        text, offsets = make_text(words, wl.seed, wl.nonascii_p)
        out["text"] = text
        out["offsets"] = offsets
    if wl.ticks:
        amax = float(arrival_sorted[-1]) if n else 0.0
        t = np.array([k * amax / wl.ticks for k in range(1, wl.ticks + 1)])
        out["tick_t"] = t
        # requests are stored in arrival order here, so each tick's pending
        # set is a prefix
        out["tick_n"] = np.searchsorted(arrival_sorted, t, side="right").astype(np.int64)
    return out


def complete(b, est_base):
    """Completion events of batch ``b`` given each request's B-free admission
    estimate ``est_base`` (float64, batch order; computed by a score call).

    Adds ``ev_est`` (the estimate the event carries), ``ev_obs`` (observed
    output tokens: the estimate times the event's drift ratio, rounded half to
    even, clipped to uint32) and ``observed`` (the same lengths per request,
    batch order), and returns ``b``. This is the serving engine's synthetic
    output model, not a stage of the method.
    """
    est_base = np.ascontiguousarray(est_base, dtype=np.float64)
    if est_base.shape != (b.n,):
        raise ValueError("est_base must hold one estimate per request")
    ev_est = est_base[b.ev_req]
    obs = np.clip(np.rint(ev_est * b.ev_ratio), 0, 2**32 - 1).astype(np.uint32)
    observed = np.empty(b.n, dtype=np.uint32)
    observed[b.ev_req] = obs
    b["ev_est"] = ev_est
    b["ev_obs"] = obs
    b["observed"] = observed
    return b


def sim_ticks(arrival, batch=32, dt=0.01, extra=16):
    """Dispatch tick times dt, 2 dt, ...: one tick per `dt` seconds (the
    batch wait), enough of them to dispatch every request in batches of
    `batch` once all have arrived, plus `extra`."""
    n = len(arrival)
    amax = float(np.max(arrival)) if n else 0.0
    k = max(int(np.ceil(amax / dt)), -(-n // batch)) + extra
    return dt * np.arange(1, k + 1, dtype=np.float64)


def text_bytes_estimate(wl):
    lo, hi = wl.words
    per_word = 6.5 * (1.0 + wl.nonascii_p * 1.5) + 2.0
    return wl.n * (lo + hi) / 2.0 * per_word
