"""The C ABI's host code (argument checks, split-KV planning, dispatch
tables, workspace sizes) built with the host compiler under AddressSanitizer
and UndefinedBehaviorSanitizer, with the kernel launchers replaced by
host-only stand-ins that check every plan (tests/host_fuzz/), and run over
random ragged batches: the queried workspace is exactly what the call
demands, and every work unit is dispatched once.  No GPU is used."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_plan_fuzz_under_asan_ubsan(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime.h")):
        pytest.skip("needs g++ and the HIP headers")
    exe = tmp_path / "plan_fuzz"
    src = [os.path.join(ROOT, "paper_2607_22663_amd", "csrc", "abi.cpp"),
           os.path.join(ROOT, "tests", "host_fuzz", "launch_stubs.cpp"),
           os.path.join(ROOT, "tests", "host_fuzz", "plan_fuzz.cpp")]
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2607_22663_amd", "csrc"), *src, "-L", os.path.join(ROCM, "lib"),
           "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    for seed in (1, 2, 3):
        r = subprocess.run([str(exe), str(seed), "4000"], capture_output=True, text=True, timeout=300)
        assert r.returncode == 0, (seed, r.stdout[-2000:], r.stderr[-4000:])
        assert "plan_fuzz ok" in r.stdout
        print(r.stdout.strip())
