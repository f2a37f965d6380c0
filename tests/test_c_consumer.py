"""The boundary from C: tests/abi_consumer.c, a C99 program that includes
include/solfp4.h and links libsolfp4.so, compiled with the host C compiler
(-Wall -Wextra -pedantic -Werror) and run without a GPU (host-only queries
and argument errors only)."""
import os
import shutil
import subprocess

import pytest

import paper_2604_06916_amd as sol

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_c_program_uses_the_boundary(tmp_path):
    libdir = os.path.dirname(sol.LIB_PATH)
    exe = tmp_path / "abi_consumer"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "abi_consumer.c"),
           "-L", libdir, "-lsolfp4", f"-Wl,-rpath,{libdir}", "-Wl,--allow-shlib-undefined",
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
