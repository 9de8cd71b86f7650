"""CPU sanitizer builds (AddressSanitizer + UndefinedBehaviorSanitizer).

1. The oracle (oracle/driftsched_ref.c) with a C driver that calls every
   function on small inputs and edge cases (tests/sanitize/oracle_checks.c).
2. The host side of the C ABI: the library's API source compiled with the
   sanitizers on its host code only, linked with the library's other objects
   and a driver that exercises every entry point's argument checks and the
   workspace-size and status functions (tests/sanitize/abi_host_checks.c).
   Those calls return before touching a GPU, so both run without one.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = "-fsanitize=address,undefined"


def run(cmd, env=None, timeout=600):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-2000:], r.stderr[-4000:])
    return r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_checks")
    run(["gcc", "-std=gnu11", "-O1", "-g", SAN, "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         "-ffp-contract=off", "-Wall", "-o", exe, os.path.join(HERE, "oracle_checks.c"),
         os.path.join(ROOT, "oracle", "driftsched_ref.c"), "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0")
    assert "ok" in run([exe], env=env)


def test_abi_host_side_under_asan_ubsan(tmp_path):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        pytest.skip("hipcc / clang++ not available")
    from paper_2606_02982_amd import build
    objs = [os.path.join(build.BUILD_DIR, os.path.splitext(s)[0] + ".o") for s in build.SOURCES
            if s != "api.hip"]
    if not all(os.path.exists(o) for o in objs):
        build.build()
    api_o = str(tmp_path / "api.o")
    flags = [f for f in build.HIP_FLAGS if f != "-O3"] + ["-O1", "-g"]
    # sanitizers on the host pass only
    for f in (SAN, "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"):
        flags += ["-Xarch_host", f]
    run([HIPCC] + flags + ["-c", os.path.join(ROOT, "paper_2606_02982_amd", "csrc", "api.hip"),
                           "-o", api_o])
    main_o = str(tmp_path / "main.o")
    run([CLANG, "-x", "c", "-O1", "-g", SAN, "-fno-sanitize-recover=all",
         "-I" + os.path.join(ROOT, "include"), "-c", os.path.join(HERE, "abi_host_checks.c"), "-o", main_o])
    exe = str(tmp_path / "abi_checks")
    run([CLANG, SAN, "-o", exe, main_o, api_o] + objs +
        ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    # the HIP runtime keeps allocations until exit: leak checks off here
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    assert "ok" in run([exe], env=env, timeout=300)
