"""ds_characterize_score_noalloc (no workspace: the library's static scratch
array) against ds_characterize_score with a workspace, bit for bit, on two
calls in a row, the second with a smaller input (the array keeps the first
call's contents), and its host-side errors."""
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


def args_for(b, n):
    text = b.text[:int(b.offsets[n])]
    return ([dev(text), dev(b.offsets[:n + 1])],
            [dev(b.category[:n]), dev(b.tenant[:n]), dev(b.group[:n]), dev(b.t_base),
             dev(b.s_tenant), torch.linspace(0.5, 1.5, b.n_groups, dtype=torch.float64,
                                             device="cuda")])


def outputs(n):
    return (torch.empty(n, dtype=torch.int32, device="cuda"),
            (torch.empty(n, dtype=torch.float64, device="cuda"),
             torch.empty(n, dtype=torch.float64, device="cuda"),
             torch.empty(n, dtype=torch.float64, device="cuda"),
             torch.empty(n, dtype=torch.uint8, device="cuda")))


def test_noalloc_equals_workspace_call(ds):
    b = wl.load("batch64k")
    for n in (b.n, 5000):          # the second call is smaller
        print("noalloc characterize_score n=%d" % n, flush=True)
        (t, o), rest = args_for(b, n)
        want_c, want = ds.characterize_score(t, o, *rest)
        c, out = outputs(n)
        got_c, got = ds.characterize_score_noalloc(t, o, *rest, counts=c, out=out)
        torch.cuda.synchronize()
        assert np.array_equal(host(got_c), host(want_c))
        assert np.array_equal(host(got_c, np.uint32), b.words[:n])
        for g, w in zip(got, want):
            assert np.array_equal(host(g), host(w))


def test_noalloc_host_errors(ds):
    b = wl.load("batch4k")
    (t, o), rest = args_for(b, 100)
    c, out = outputs(100)
    # DS_VALIDATE is refused (flags must be 0)
    p = ds.ScoreParams(1024.0, 128.0, 512.0)
    st = ds.lib.ds_characterize_score_noalloc(
        ds._ptr(t), t.numel(), ds._ptr(o), 100, ds._ptr(c), ds._ptr(rest[0]), ds._ptr(rest[1]),
        ds._ptr(rest[2]), ds._ptr(rest[3]), 4, ds._ptr(rest[4]), rest[4].numel(), ds._ptr(rest[5]),
        rest[5].numel(), p, ds._ptr(out[0]), ds._ptr(out[1]), ds._ptr(out[2]), ds._ptr(out[3]),
        ds.DS_VALIDATE, ds._stream())
    assert st == -2
