"""The library's host runtime under AddressSanitizer and UBSan, on the CPU.

tests/native/runtime_host_check.cpp compiles the runtime source
(paper_2411_17866_amd/csrc/dsm_runtime.cpp) with g++ against stubs of the HIP
calls the runtime makes (device count and current device, copy, stream sync,
error string), of the static-scratch lookup and of the kernel launchers, so
the whole C ABI runs without a GPU.  Its checks are:
  * dsm_layout on 3000 random valid and invalid problems, in the three
    replica layouts;
  * the uploaded chunk table;
  * the blocked layouts' addressing: every piece inside one block, and every
    element of every copy at its own slot of the allocation;
  * the randomized sign's bound words in the workspace;
  * the Algorithm 1 state machine, with the layouts and XCD map of each launch;
  * the replica source of each local launch, fresh or stale;
  * dsm_init_static: the static scratch, its limit, one context per device;
  * the fp32 host coefficients against long double;
  * every error path.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2411_17866_amd", "csrc")
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")


def test_runtime_host_logic_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no g++")
    if not os.path.exists(os.path.join(ROCM_INCLUDE, "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not installed")
    exe = str(tmp_path / "runtime_host_check")
    # Host code only (g++, no HIP source on this line): the sanitizer runtime
    # is linked statically so it comes first whatever else the process loads.
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-static-libasan",
           "-Wall", "-Wextra", "-Werror", "-Wno-unused-parameter",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM_INCLUDE}", f"-I{os.path.join(ROOT, 'include')}",
           f"-I{CSRC}", os.path.join(ROOT, "tests", "native", "runtime_host_check.cpp"),
           os.path.join(CSRC, "dsm_runtime.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "all checks passed" in r.stdout
