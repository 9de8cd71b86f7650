"""The C ABI library: it loads, exports every entry point the header
declares, and rejects bad host arguments before touching a device (these
calls return before any HIP call, so they run without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "driftsched.h")


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ds_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(ds):
    names = declared_functions()
    assert names == ["ds_calibrate", "ds_calibrate_ex", "ds_characterize", "ds_characterize_score",
                     "ds_characterize_score_noalloc", "ds_class_histogram", "ds_error_stats", "ds_order", "ds_order_multi",
                     "ds_read_bandwidth", "ds_score", "ds_simulate", "ds_simulate_multi", "ds_status_string", "ds_version",
                     "ds_workspace_bytes"]
    for name in names:
        assert hasattr(ds.lib, name), name


def test_status_strings(ds):
    for code in range(-8, 1):
        s = ds.status_string(code)
        assert s and s != "unknown status"
    assert ds.status_string(-99) == "unknown status"
    assert ds.lib.ds_version() == 10000


def test_workspace_sizes(ds):
    for op in range(8):
        sizes = [ds.workspace_bytes(op, n, 64) for n in (0, 1, 4096, 65536, 1 << 20)]
        assert all(s >= 256 for s in sizes)
        assert sizes == sorted(sizes)
    assert ds.workspace_bytes(ds.OP_SCORE, 1 << 20) == 256
    assert ds.workspace_bytes(ds.OP_CLASS_HIST, 1 << 20) == 256
    # error statistics: sums for every group and for all events
    assert ds.workspace_bytes(ds.OP_ERROR_STATS, 10, 7) >= 256 + 4 * 8 * 8
    # several tick loops: the third argument is the number of runs (1..256)
    for n in (1, 4096, 65536):
        assert ds.workspace_bytes(ds.OP_SIMULATE_MULTI, n, 1) == ds.workspace_bytes(ds.OP_SIMULATE, n)
        assert ds.workspace_bytes(ds.OP_SIMULATE_MULTI, n, 8) > ds.workspace_bytes(ds.OP_SIMULATE_MULTI, n, 2)
        assert ds.workspace_bytes(ds.OP_SIMULATE_MULTI, n, 0) == 0
        assert ds.workspace_bytes(ds.OP_SIMULATE_MULTI, n, ds.SIM_MAX_RUNS) > 0
        assert ds.workspace_bytes(ds.OP_SIMULATE_MULTI, n, ds.SIM_MAX_RUNS + 1) == 0


P = ctypes.c_void_p
NULL = None
FAKE = P(0x1000)          # never dereferenced: every call below fails host checks
FAKE_WS = P(0x100000)


def test_characterize_host_errors(ds):
    f = ds.lib.ds_characterize
    assert f(NULL, 0, NULL, 0, NULL, NULL, 0, 0, NULL) == 0          # n == 0: nothing to do
    assert f(FAKE, 16, NULL, 4, FAKE, FAKE_WS, 1 << 30, 0, NULL) == -1
    assert f(NULL, 16, FAKE, 4, FAKE, FAKE_WS, 1 << 30, 0, NULL) == -1
    assert f(P(0x1001), 16, FAKE, 4, FAKE, FAKE_WS, 1 << 30, 0, NULL) == -7
    assert f(FAKE, 16, FAKE, 4, FAKE, FAKE_WS, 16, 0, NULL) == -4      # short workspace
    assert f(FAKE, 16, FAKE, 4, FAKE, P(0x100001), 1 << 30, 0, NULL) == -4
    assert f(FAKE, 16, FAKE, 0xFFFFFFFF, FAKE, FAKE_WS, 1 << 30, 0, NULL) == -3


def test_calibrate_host_errors(ds):
    f = ds.lib.ds_calibrate
    assert f(FAKE, FAKE, FAKE, 10, 1.5, 4, FAKE, NULL, FAKE_WS, 1 << 30, 0, NULL) == -2
    assert f(FAKE, FAKE, FAKE, 10, -0.1, 4, FAKE, NULL, FAKE_WS, 1 << 30, 0, NULL) == -2
    assert f(FAKE, FAKE, FAKE, 10, float("nan"), 4, FAKE, NULL, FAKE_WS, 1 << 30, 0, NULL) == -2
    assert f(FAKE, FAKE, FAKE, 10, 0.1, 0, FAKE, NULL, FAKE_WS, 1 << 30, 0, NULL) == -2
    assert f(FAKE, FAKE, FAKE, (1 << 30) + 1, 0.1, 4, FAKE, NULL, FAKE_WS, 1 << 40, 0, NULL) == -3
    assert f(NULL, FAKE, FAKE, 10, 0.1, 4, FAKE, NULL, FAKE_WS, 1 << 30, 0, NULL) == -1
    assert f(FAKE, FAKE, FAKE, 10, 0.1, 4, FAKE, NULL, FAKE_WS, 100, 0, NULL) == -4
    assert f(FAKE, FAKE, FAKE, 0, 0.1, 4, FAKE, NULL, NULL, 0, 0, NULL) == 0


def test_score_host_errors(ds):
    f = ds.lib.ds_score
    good = ds.ScoreParams(1024.0, 128.0, 512.0)
    bad = ds.ScoreParams(0.0, 128.0, 512.0)
    args = [FAKE] * 4 + [FAKE, 4, FAKE, 3, FAKE, 3]
    assert f(10, *args, ctypes.byref(bad), NULL, FAKE, FAKE, FAKE, NULL, 0, 0, NULL) == -2
    assert f(10, *args, None, NULL, FAKE, FAKE, FAKE, NULL, 0, 0, NULL) == -1
    assert f(10, NULL, *args[1:], ctypes.byref(good), NULL, FAKE, FAKE, FAKE, NULL, 0, 0, NULL) == -1
    assert f(10, *args, ctypes.byref(good), NULL, FAKE, FAKE, FAKE, NULL, 0, 1, NULL) == -4
    assert f(0, *args, ctypes.byref(good), NULL, FAKE, FAKE, FAKE, NULL, 0, 0, NULL) == 0


def test_order_host_errors(ds):
    f = ds.lib.ds_order
    p = ds.order_params()
    ws = 1 << 40
    assert f(7, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(p), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    q = ds.order_params(n_tiers=0)
    assert f(0, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    q = ds.order_params(n_tiers=17)
    assert f(0, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    q = ds.order_params(weights=(1, 0, 1))
    assert f(2, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    q = ds.order_params(aging_rate=-1.0)
    assert f(4, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    # the smooth interleaving: a known mode, weights summing to at most 1024
    q = ds.order_params(weighted_mode=3)
    assert f(2, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    q = ds.order_params(weights=(4000, 1, 1), weighted_mode="stride")    # no bound for stride
    assert f(2, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, 64, 0, NULL) == -4
    q = ds.order_params(weights=(1000, 24, 1), weighted_mode="smooth")
    assert f(2, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -2
    q = ds.order_params(weights=(1000, 23, 1), weighted_mode="smooth")   # sum 1024: accepted
    assert f(2, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, 64, 0, NULL) == -4
    q = ds.order_params(weights=(4000, 1, 1), weighted_mode="blocked")  # no bound when blocked
    assert f(2, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, 64, 0, NULL) == -4
    q = ds.order_params(weights=(4000, 1, 1), weighted_mode=7)           # only Weighted reads the mode
    assert f(0, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(q), FAKE, NULL, FAKE_WS, 64, 0, NULL) == -4
    assert f(3, 10, FAKE, FAKE, NULL, NULL, ctypes.byref(p), FAKE, NULL, FAKE_WS, ws, 0, NULL) == -1
    assert f(0, (1 << 30) + 1, FAKE, FAKE, NULL, NULL, ctypes.byref(p), FAKE, NULL, FAKE_WS, ws, 0,
             NULL) == -3
    assert f(0, 10, FAKE, FAKE, NULL, NULL, ctypes.byref(p), FAKE, NULL, FAKE_WS, 64, 0, NULL) == -4
    assert f(0, 0, NULL, NULL, NULL, NULL, ctypes.byref(p), NULL, NULL, NULL, 0, 0, NULL) == 0


def test_order_multi_host_errors(ds):
    f = ds.lib.ds_order_multi
    p = ds.order_params()
    ws = 1 << 40
    perms = (ctypes.c_void_p * 5)(0x1000, 0x1000, 0x1000, 0x1000, 0x1000)
    nulls = (ctypes.c_void_p * 5)()
    assert f(0, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(p), perms, NULL, FAKE_WS, ws, 0, NULL) == -2
    assert f(0x20, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(p), perms, NULL, FAKE_WS, ws, 0, NULL) == -2
    assert f(0x1F, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(p), NULL, NULL, FAKE_WS, ws, 0, NULL) == -1
    assert f(0x03, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(p), nulls, NULL, FAKE_WS, ws, 0, NULL) == -1
    assert f(0x08, 10, FAKE, FAKE, NULL, NULL, ctypes.byref(p), perms, NULL, FAKE_WS, ws, 0, NULL) == -1
    need = ds.workspace_bytes(ds.OP_ORDER_MULTI, 10)
    assert need > ds.workspace_bytes(ds.OP_ORDER, 10)
    assert f(0x1F, 10, FAKE, FAKE, FAKE, NULL, ctypes.byref(p), perms, NULL, FAKE_WS, need - 1, 0,
             NULL) == -4


def test_calibrate_ex_host_errors(ds):
    f = ds.lib.ds_calibrate_ex
    ws = 1 << 30
    assert f(FAKE, FAKE, FAKE, 10, 1.5, 4, FAKE, NULL, NULL, FAKE_WS, ws, 0, NULL) == -2
    assert f(FAKE, FAKE, FAKE, 10, 0.1, 4, FAKE, NULL, P(0x1004), FAKE_WS, ws, 0, NULL) == -7
    assert f(FAKE, NULL, FAKE, 10, 0.1, 4, FAKE, NULL, FAKE, FAKE_WS, ws, 0, NULL) == -1
    assert f(FAKE, FAKE, FAKE, 0, 0.1, 4, FAKE, NULL, NULL, NULL, 0, 0, NULL) == 0


def test_error_stats_host_errors(ds):
    f = ds.lib.ds_error_stats
    ws = 1 << 30
    # group and n_groups go together
    assert f(10, FAKE, NULL, FAKE, FAKE, 0, FAKE, FAKE_WS, ws, 0, NULL) == -2
    assert f(10, FAKE, NULL, FAKE, NULL, 3, FAKE, FAKE_WS, ws, 0, NULL) == -2
    assert f(10, FAKE, NULL, FAKE, FAKE, (1 << 20) + 1, FAKE, FAKE_WS, ws, 0, NULL) == -3
    assert f((1 << 30) + 1, FAKE, NULL, FAKE, NULL, 0, FAKE, FAKE_WS, ws, 0, NULL) == -3
    assert f(10, NULL, NULL, FAKE, NULL, 0, FAKE, FAKE_WS, ws, 0, NULL) == -1
    assert f(10, FAKE, NULL, FAKE, NULL, 0, NULL, FAKE_WS, ws, 0, NULL) == -1
    assert f(10, P(0x1004), NULL, FAKE, NULL, 0, FAKE, FAKE_WS, ws, 0, NULL) == -7
    assert f(10, FAKE, NULL, FAKE, FAKE, 5, FAKE, FAKE_WS, 64, 0, NULL) == -4


def test_class_histogram_host_errors(ds):
    f = ds.lib.ds_class_histogram
    assert f(10, FAKE, 0, FAKE, FAKE, NULL, 0, 0, NULL) == -2
    assert f(10, FAKE, 257, FAKE, FAKE, NULL, 0, 0, NULL) == -2
    assert f(10, NULL, 4, FAKE, FAKE, NULL, 0, 0, NULL) == -1
    assert f(10, FAKE, 4, FAKE, NULL, NULL, 0, 0, NULL) == -1
    assert f(10, FAKE, 4, FAKE, P(0x1002), NULL, 0, 0, NULL) == -7
    assert f(10, FAKE, 4, FAKE, FAKE, NULL, 0, 1, NULL) == -4     # DS_VALIDATE needs a workspace


def test_simulate_host_errors(ds):
    f = ds.lib.ds_simulate
    ws = 1 << 40

    # every call below must fail a host check (none may reach a launch)
    def call(params, n=10, n_cat=4, n_tenants=2, n_groups=3, tick_t=FAKE, n_ticks=5, seq=FAKE,
             nd=FAKE, wsb=ws, arrival=FAKE):
        st = f(n, arrival, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, n_cat, FAKE, n_tenants,
               n_groups, tick_t, n_ticks, ctypes.byref(params) if params is not None else None,
               FAKE, seq, FAKE, nd, FAKE_WS, wsb, 0, NULL)
        assert st != 0
        return st

    ok = ds.sim_params("sjf")
    assert call(None) == -1
    assert call(ds.sim_params(5)) == -2
    assert call(ds.sim_params("fifo", batch=0)) == -2
    assert call(ds.sim_params("fifo", batch=1025)) == -2
    assert call(ds.sim_params("fifo", alpha=1.5)) == -2
    assert call(ds.sim_params("fifo", f_ref=0.0)) == -2
    assert call(ds.sim_params("weighted", weights=(1, 0, 1))) == -2
    assert call(ds.sim_params("weighted", weighted_mode=3)) == -2
    assert call(ds.sim_params("weighted", weights=(1020, 4, 1), weighted_mode="smooth")) == -2
    assert call(ds.sim_params("aging", aging_rate=-1.0)) == -2
    assert call(ds.sim_params("fifo", n_tiers=0)) == -2
    assert call(ok, n_cat=0) == -2 and call(ok, n_cat=257) == -2
    assert call(ok, n_tenants=0) == -2 and call(ok, n_groups=0) == -2
    assert call(ok, n=(1 << 30) + 1) == -3
    assert call(ok, n_ticks=1 << 31) == -3
    assert call(ok, nd=NULL) == -1 and call(ok, seq=NULL) == -1
    assert call(ok, tick_t=NULL) == -1
    assert call(ok, arrival=P(0x1004)) == -7
    assert call(ok, wsb=ds.workspace_bytes(ds.OP_SIMULATE, 10) - 1) == -4
    # t_now is not used: each tick ages to its own time
    assert call(ds.sim_params("aging", t_now=float("nan")), wsb=64) == -4


def test_characterize_score_host_errors(ds):
    f = ds.lib.ds_characterize_score
    good = ds.ScoreParams(1024.0, 128.0, 512.0)
    bad = ds.ScoreParams(0.0, 128.0, 512.0)
    # category, tenant, group, t_base, n_cat, s_tenant, n_tenants, state, n_groups
    sc = [FAKE, FAKE, FAKE, FAKE, 4, FAKE, 3, FAKE, 3]
    outs = [NULL, FAKE, FAKE, FAKE]   # est_base, est, budget, class
    ws = 1 << 30
    assert f(FAKE, 16, FAKE, 4, FAKE, *sc, ctypes.byref(bad), *outs, FAKE_WS, ws, 0, NULL) == -2
    assert f(FAKE, 16, FAKE, 4, FAKE, *sc, None, *outs, FAKE_WS, ws, 0, NULL) == -1
    assert f(FAKE, 16, NULL, 4, FAKE, *sc, ctypes.byref(good), *outs, FAKE_WS, ws, 0, NULL) == -1
    assert f(FAKE, 16, FAKE, 4, FAKE, NULL, *sc[1:], ctypes.byref(good), *outs, FAKE_WS, ws, 0, NULL) == -1
    assert f(FAKE, 16, FAKE, 4, FAKE, *sc[:4], 0, *sc[5:], ctypes.byref(good), *outs, FAKE_WS, ws, 0,
             NULL) == -2
    assert f(P(0x1001), 16, FAKE, 4, FAKE, *sc, ctypes.byref(good), *outs, FAKE_WS, ws, 0, NULL) == -7
    assert f(FAKE, 16, FAKE, 4, FAKE, *sc, ctypes.byref(good), *outs, FAKE_WS, 16, 0, NULL) == -4
    assert f(FAKE, 16, FAKE, 0xFFFFFFFF, FAKE, *sc, ctypes.byref(good), *outs, FAKE_WS, ws, 0, NULL) == -3
    assert f(NULL, 0, NULL, 0, NULL, *sc, ctypes.byref(good), *outs, NULL, 0, 0, NULL) == 0


def test_characterize_score_noalloc_host_errors(ds):
    # checked before anything touches a GPU
    P = ds.ScoreParams(1024.0, 128.0, 512.0)
    x = ctypes.c_void_p(256)
    call = lambda n, flags, params=P: ds.lib.ds_characterize_score_noalloc(
        x, 16, x, n, x, x, x, x, x, 4, x, 3, x, 3, params, None, x, x, x, flags, None)
    assert call(ds.NOALLOC_MAX_PROMPTS + 1, 0) == -3         # above the scratch array's limit
    assert call(10, 1) == -2                                  # DS_VALIDATE refused
    assert call(0, 0) == 0                                    # empty batch
    assert call(10, 0, None) == -1
    assert ds.workspace_bytes(ds.OP_CHARACTERIZE, ds.NOALLOC_MAX_PROMPTS) <= 4456960


def test_read_bandwidth_host_errors(ds):
    f = ds.lib.ds_read_bandwidth
    assert f(FAKE, 17, FAKE, NULL) == -2      # not a multiple of 16
    assert f(NULL, 32, FAKE, NULL) == -1
    assert f(FAKE, 32, NULL, NULL) == -1
    assert f(P(0x1008), 32, FAKE, NULL) == -7  # not 16-byte aligned
    assert f(FAKE, 32, P(0x1002), NULL) == -7


def test_param_struct_layouts_match_the_header(ds, tmp_path):
    # the binding's ctypes structures have the C header's sizes and field
    # offsets (gcc compiles a program that prints them)
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    structs = {"ds_score_params": ds.ScoreParams, "ds_order_params": ds.OrderParams,
               "ds_sim_params": ds.SimParams}
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "driftsched.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append('printf("%s %%zu\\n", sizeof(%s));' % (cname, cname))
        for fname, _ in cls._fields_:
            lines.append('printf("%s.%s %%zu\\n", offsetof(%s, %s));' % (cname, fname, cname, fname))
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run(["gcc", "-std=c99", "-I", inc, str(src), "-o", str(exe)], check=True)
    got = dict(line.split() for line in subprocess.run([str(exe)], check=True, capture_output=True,
                                                        text=True).stdout.splitlines())
    for cname, cls in structs.items():
        assert int(got[cname]) == ctypes.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert int(got["%s.%s" % (cname, fname)]) == getattr(cls, fname).offset, (cname, fname)
