"""The C ABI's host runtime under AddressSanitizer and UndefinedBehaviorSanitizer.

csrc/api.cpp is compiled for the host alone with clang (no device code),
linked with stand-ins for the HIP runtime and the kernel launchers
(tests/host/hip_host_stub.cpp: device memory is host memory, launches only
touch the bounds of the regions the real kernels access and check index
tables), and driven through include/dif.h by tests/host/harness.cpp:
config and mask validation, plans of both kinds over seeded masks with
empty and gated-off layers, workspace and text-cache carving at ragged
token counts, the timestep bound to a plan (Sec. 3.1 / Sec. 3.2: the
structure g_{t_i} belongs to t_i), rollouts, FFN reorder, hard gates, the
operator entry points and kernel timing.  Any out-of-bounds access, leak or
undefined behaviour fails the run.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang++"


@pytest.mark.skipif(not os.path.exists(CLANG), reason="ROCm clang++ not installed")
def test_host_runtime_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "harness"
    cmd = [CLANG, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           os.path.join(ROOT, "paper_2607_06631_amd", "csrc", "api.cpp"),
           os.path.join(ROOT, "tests", "host", "hip_host_stub.cpp"),
           os.path.join(ROOT, "tests", "host", "harness.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    print(r.stdout)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "harness: all cases passed" in r.stdout
    shutil.rmtree(tmp_path, ignore_errors=True)
