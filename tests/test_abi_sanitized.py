"""The C ABI's host layer (argument validation, workspace sizing, the dispatch
decisions of api.cpp and plan.cpp) built with a host compiler under
AddressSanitizer and UndefinedBehaviorSanitizer, with the kernel launchers and
the HIP runtime functions it calls replaced by host stand-ins
(tests/asan/hip_stubs.cpp), and driven through every entry point's checks by
tests/asan/abi_validation.cpp."""

import os
import shutil
import subprocess

import pytest

from _helpers import ROOT

CSRC = os.path.join(ROOT, "paper_2410_01651_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "asan")


def test_validation_layer_under_sanitizers(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = tmp_path / "abi_validation"
    sanitize = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
    cmd = [cxx, "-std=c++17", "-O1", "-g", *sanitize, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "plan.cpp"),
           os.path.join(HERE, "hip_stubs.cpp"), os.path.join(HERE, "abi_validation.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env)
    assert r.returncode == 0 and r.stdout.strip() == "OK", (r.stdout + r.stderr)[-4000:]
