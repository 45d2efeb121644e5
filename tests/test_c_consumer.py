"""include/noble.h is plain C: a C99 program that includes it builds with
-Wall -Wextra -pedantic -Werror, links against libnoble.so and passes its
host-side checks (tests/c/abi_consumer.c); the header also compiles as C++."""

import os
import shutil
import subprocess

import pytest

from paper_2603_06492_amd import noble

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")


def _compiler(name):
    cc = shutil.which(name)
    if cc is None:
        pytest.skip(f"{name} not found")
    return cc


def test_c99_consumer_builds_links_and_runs(tmp_path):
    cc = _compiler("gcc")
    noble.lib()   # raises if the library has not been built
    lib_dir = os.path.dirname(noble.LIB_PATH)
    exe = tmp_path / "abi_consumer"
    cmd = [cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", INCLUDE,
           os.path.join(ROOT, "tests", "c", "abi_consumer.c"), "-o", str(exe),
           "-L", lib_dir, "-lnoble", f"-Wl,-rpath,{lib_dir}", "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0 and run.stdout.strip() == "ok", run.stdout + run.stderr


def test_header_compiles_as_cpp(tmp_path):
    cxx = _compiler("g++")
    src = tmp_path / "h.cpp"
    src.write_text('#include "noble.h"\nstatic_assert(sizeof(noble_linear_desc) == 48, "desc layout");\n'
                   "int main() { return noble_abi_version() == NOBLE_ABI_VERSION ? 0 : 1; }\n")
    res = subprocess.run([cxx, "-std=c++17", "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only",
                          "-I", INCLUDE, str(src)], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
