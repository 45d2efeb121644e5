"""The host side of libnoble (argument validation, workspace sizing, the
weight-gradient planner, the recipe's host calls) built with
AddressSanitizer and UndefinedBehaviorSanitizer, and driven on the CPU by
the C99 consumer (tests/c/abi_consumer.c) and a sweep over shapes up to the
ABI's limits (tests/c/host_sweep.c).  Only host code is instrumented
(each -fsanitize= follows -Xarch_host); the device code is the ordinary
build.  Any memory error or undefined behaviour aborts a run."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_06492_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
LLVM = "/opt/rocm/lib/llvm/bin/clang"
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not found")


@pytest.fixture(scope="module")
def asan_lib(tmp_path_factory):
    if not os.path.exists(LLVM):
        pytest.skip("ROCm clang not found")
    d = tmp_path_factory.mktemp("asan")
    lib = d / "libnoble.so"
    host_san = [x for f in SAN for x in ("-Xarch_host", f)]
    cmd = [_hipcc(), "-O1", "-g", "-std=c++20", "--offload-arch=gfx950", "-fPIC", "-shared", "-munsafe-fp-atomics",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san,
           "-I", INCLUDE, "-I", CSRC, os.path.join(CSRC, "noble_api.hip"), "-o", str(lib)]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    return d


def _run(asan_lib, src):
    exe = asan_lib / os.path.splitext(os.path.basename(src))[0]
    cmd = [LLVM, "-std=c99", "-g", *SAN, "-Wall", "-Wextra", "-Werror", "-I", INCLUDE, src, "-o", str(exe),
           "-L", str(asan_lib), "-lnoble", f"-Wl,-rpath,{asan_lib}", "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600, env=env)
    assert run.returncode == 0, run.stdout + run.stderr[-4000:]
    return run.stdout.strip()


def test_consumer_under_sanitizers(asan_lib):
    assert _run(asan_lib, os.path.join(ROOT, "tests", "c", "abi_consumer.c")) == "ok"


def test_shape_sweep_under_sanitizers(asan_lib):
    out = _run(asan_lib, os.path.join(ROOT, "tests", "c", "host_sweep.c"))
    assert out.startswith("ok ") and int(out.split()[1]) > 10000, out
