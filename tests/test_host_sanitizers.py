"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):
the scaling-policy library (paper_2606_29207_amd/csrc/kf_policy.cpp, plain
C++) is compiled with both sanitizers and driven by tests/c/policy_stress.c
through every entry point of include/kf_policy.h, over random batches, with
every output array allocated at exactly the capacity it is passed with, and
through its capacity refusals and invalid-argument paths.  Any out-of-bounds
access, leak, use after free or undefined behaviour fails the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                    reason="needs gcc and g++")
def test_policy_library_under_asan_and_ubsan(tmp_path):
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    inc = ["-I", os.path.join(ROOT, "include")]
    obj = tmp_path / "kf_policy.o"
    exe = tmp_path / "policy_stress"
    steps = [
        ["g++", "-std=c++17", "-O1", "-g", "-Wall", *san, *inc, "-c",
         os.path.join(ROOT, "paper_2606_29207_amd", "csrc", "kf_policy.cpp"), "-o", str(obj)],
        ["gcc", "-std=c99", "-O1", "-g", "-Wall", "-Wextra", *san, *inc, "-c",
         os.path.join(ROOT, "tests", "c", "policy_stress.c"), "-o", str(tmp_path / "stress.o")],
        ["g++", *san, str(tmp_path / "stress.o"), str(obj), "-o", str(exe), "-lm"],
    ]
    for cmd in steps:
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, " ".join(cmd) + "\n" + res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    run = subprocess.run([str(exe), "300"], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0 and "policy_stress ok" in run.stdout, run.stdout + run.stderr[-4000:]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_api_layer_under_asan_and_ubsan(tmp_path):
    """The C-ABI layer (kf_api.cpp: argument checks, launch planning and
    workspace sizing) built with g++ under both sanitizers against a host-only
    HIP test double, its kernel launchers replaced by checkers
    (tests/c/api_stress.cpp): valid calls, one broken argument at a time,
    arbitrary arguments, and the plan and workspace queries over random and
    extreme sizes on devices of 1 to 1024 compute units."""
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    inc = ["-I", os.path.join(ROOT, "tests", "c", "hipstub"), "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2606_29207_amd", "csrc")]
    exe = tmp_path / "api_stress"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall", *san, *inc,
           os.path.join(ROOT, "paper_2606_29207_amd", "csrc", "kf_api.cpp"),
           os.path.join(ROOT, "tests", "c", "api_stress.cpp"), "-o", str(exe), "-lm"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, " ".join(cmd) + "\n" + res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    run = subprocess.run([str(exe), "400"], capture_output=True, text=True, timeout=600, env=env)
    assert run.returncode == 0 and "api_stress ok" in run.stdout, run.stdout + run.stderr[-4000:]
