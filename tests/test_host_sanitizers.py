"""The library's host code built host-only under sanitizers, on the CPU.

The planners, the validators, the kernel entry points' host-side error paths, the MPU planner and
the hint index are compiled with g++ (no device code) together with test-only stand-ins for the GPU
launchers, and driven by seeded randomized inputs:

* address + undefined-behaviour sanitizers over ``tests/native/host_fuzz.cpp`` (every accepted
  attention plan's work list is checked for exact coverage; every status against a restatement of
  the validation rules);
* thread sanitizer over ``tests/native/hints_threads.cpp`` (concurrent add / detach / probe of the
  sharded hint index).

The builds go to a temporary directory; nothing is written into the tree.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35263_amd", "csrc")
NATIVE = os.path.join(ROOT, "tests", "native")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HOST_SOURCES = [os.path.join(CSRC, f) for f in ("host.cpp", "kda_host.cpp", "mpu.cpp", "hints.cpp")]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir(os.path.join(ROCM, "include")),
                                reason="needs g++ and the ROCm headers")


def _build(out, sources, sanitize, link_hip=True):
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", f"-fsanitize={sanitize}",
           "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-I", os.path.join(ROCM, "include"), *sources, "-o", out, "-pthread"]
    if link_hip:
        cmd += ["-L", os.path.join(ROCM, "lib"), "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-lamdhip64"]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, f"build failed:\n{' '.join(cmd)}\n{res.stderr[-4000:]}"


def _run(exe, args, extra_env):
    env = dict(os.environ)
    env.update(extra_env)
    res = subprocess.run([exe, *args], capture_output=True, text=True, timeout=600, env=env)
    assert res.returncode == 0, f"{exe} {args} failed ({res.returncode}):\n{res.stdout[-2000:]}\n{res.stderr[-6000:]}"
    assert "runtime error" not in res.stderr and "Sanitizer" not in res.stderr, res.stderr[-6000:]
    return res.stdout


def test_host_code_under_address_and_undefined_behaviour_sanitizers():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "host_fuzz")
        _build(exe, HOST_SOURCES + [os.path.join(NATIVE, "launch_stubs.cpp"), os.path.join(NATIVE, "host_fuzz.cpp")],
               "address,undefined")
        for seed in ("1", "2", "3"):
            out = _run(exe, ["1500", seed], {"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0",
                                             "UBSAN_OPTIONS": "print_stacktrace=1"})
            assert "host_fuzz ok" in out


def test_hint_index_under_thread_sanitizer():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "hints_threads")
        _build(exe, HOST_SOURCES + [os.path.join(NATIVE, "launch_stubs.cpp"), os.path.join(NATIVE, "hints_threads.cpp")],
               "thread")
        out = _run(exe, ["40"], {"TSAN_OPTIONS": "halt_on_error=1"})
        assert "hints_threads ok" in out
