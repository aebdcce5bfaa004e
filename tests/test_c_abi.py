"""The C ABI from plain C (no GPU): include/kf.h and include/kf_policy.h
compile as C99 with gcc, and a C program linked against libkf.so runs the
host entry points (tests/c/abi_smoke.c)."""
import os
import shutil
import subprocess

import pytest

from paper_2606_29207_amd import kf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c_client_builds_and_runs(tmp_path):
    if not os.path.exists(kf._LIB_PATH):
        from paper_2606_29207_amd import build
        build.build()
    exe = tmp_path / "abi_smoke"
    libdir = os.path.dirname(kf._LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_smoke.c"), "-o", str(exe),
           "-L", libdir, "-l:libkf.so", f"-Wl,-rpath,{libdir}", "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0 and "abi_smoke ok" in run.stdout, run.stdout + run.stderr
