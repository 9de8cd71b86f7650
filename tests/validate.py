"""Validation of the float-keyed orders (SJF, Aging).

When the budgets or aged scores of the two sides agree only within the
calibration tolerance, near-ties may fall either way, so the GPU permutation
is checked for what is unique rather than for equality:

1. it is a permutation of 0..n-1;
2. each GPU key agrees with the oracle's within 1e-12 relative
   (|gpu - oracle| <= 1e-12 * max(|oracle|, scale));
3. it is sorted by (GPU key, FIFO rank) exactly, the FIFO rank being the
   position of a request in the order of (arrival, index): every policy
   breaks ties by it;
4. the number of positions where it differs from the oracle's permutation
   is returned (0 when the keys are bit-identical).
"""
import numpy as np

KEY_RTOL = 1e-12


def fifo_rank(arrival):
    n = len(arrival)
    a = np.asarray(arrival, np.float64) + 0.0          # -0.0 equals +0.0
    order = np.lexsort((np.arange(n), a))
    rank = np.empty(n, np.int64)
    rank[order] = np.arange(n)
    return rank


def check_float_order(perm, key, want_perm, want_key, arrival, scale):
    perm = np.asarray(perm).astype(np.int64)
    key = np.asarray(key, np.float64)
    want_key = np.asarray(want_key, np.float64)
    n = len(arrival)
    assert perm.shape == (n,), "permutation has the wrong length"
    seen = np.zeros(n, bool)
    assert perm.min(initial=0) >= 0 and perm.max(initial=-1) < n, "index out of range"
    seen[perm] = True
    assert seen.all(), "not a permutation"
    tol = KEY_RTOL * np.maximum(np.abs(want_key), scale)
    bad = ~(np.abs(key - want_key) <= tol)
    assert not bad.any(), "%d keys differ beyond 1e-12 (first at %d: %r vs %r)" % (
        bad.sum(), np.argmax(bad), key[np.argmax(bad)], want_key[np.argmax(bad)])
    f = fifo_rank(arrival)
    k = key[perm] + 0.0
    r = f[perm]
    ok = (k[1:] > k[:-1]) | ((k[1:] == k[:-1]) & (r[1:] > r[:-1]))
    assert ok.all(), "not sorted by (key, FIFO rank) at position %d" % (np.argmin(ok) + 1)
    return int((perm != np.asarray(want_perm).astype(np.int64)).sum())
