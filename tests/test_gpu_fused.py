"""Stages 1 and 3 fused (ds_characterize_score) on the GPU: bit for bit the
results of ds_characterize followed by ds_score, and the oracle's counts."""
import numpy as np
import pytest
import torch

from tests import wl
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def separate_and_fused(ds, text, offsets, cat, ten, grp, tb, s, state, **kw):
    args = [dev(np.asarray(cat, np.uint8)), dev(np.asarray(ten, np.uint32)), dev(np.asarray(grp, np.uint32)),
            dev(np.asarray(tb, np.float64)), dev(np.asarray(s, np.float64)), dev(np.asarray(state, np.float64))]
    t, o = dev(text), dev(offsets)
    counts = ds.characterize(t, o)
    sep = [counts] + list(ds.score(counts, *args, **kw))
    c2, out = ds.characterize_score(t, o, *args, **kw)
    fused = [c2] + list(out)
    return [None if x is None else host(x) for x in sep], [None if x is None else host(x) for x in fused]


@pytest.mark.parametrize("name", ["batch4k", "batch64k"])
def test_workload_equals_separate_calls(ds, oracle, name):
    b = wl.load(name)
    print("fused characterize+score %s n=%d" % (name, b.n), flush=True)
    st, _ = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, 0.1, np.ones(b.n_groups), False)
    sep, fused = separate_and_fused(ds, b.text, b.offsets, b.category, b.tenant, b.group, b.t_base,
                                    b.s_tenant, st)
    assert np.array_equal(fused[0].view(np.uint32), b.words)
    for g, w in zip(fused, sep):
        assert np.array_equal(g, w)


def test_edge_prompts_and_no_est_base(ds, oracle):
    # empty prompts, whitespace-only prompts, a multi-byte separator, a
    # prompt at the end of the buffer; est_base not requested
    prompts = [b"", b"one two", b"   ", "a　b c".encode(), b"x", b"", b"\tlast words here "]
    text = np.frombuffer(b"".join(prompts), np.uint8).copy()
    offsets = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.uint64)
    n = len(prompts)
    rng = np.random.default_rng(5)
    cat, ten, grp = rng.integers(0, 4, n), rng.integers(0, 3, n), rng.integers(0, 2, n)
    sep, fused = separate_and_fused(ds, text, offsets, cat, ten, grp, [100.0, 200.0, 50.0, 400.0],
                                    [1.0, 1.5, 0.5], [0.9, 1.2], want_est_base=False)
    want = [len(p.decode("utf-8", "surrogateescape").split()) for p in prompts]
    assert fused[0].view(np.uint32).tolist() == want
    assert fused[1] is None and sep[1] is None
    for g, w in zip(fused[2:], sep[2:]):
        assert np.array_equal(g, w)


def test_validate_rejects_bad_group(ds):
    b = wl.load("batch4k")
    grp = np.asarray(b.group, np.uint32).copy()
    grp[7] = b.n_groups   # out of range
    args = [dev(np.asarray(b.category, np.uint8)), dev(np.asarray(b.tenant, np.uint32)), dev(grp),
            dev(np.asarray(b.t_base, np.float64)), dev(np.asarray(b.s_tenant, np.float64)),
            torch.ones(b.n_groups, dtype=torch.float64, device="cuda")]
    with pytest.raises(ds.DriftSchedError):
        ds.characterize_score(dev(b.text), dev(b.offsets), *args, validate=True)
