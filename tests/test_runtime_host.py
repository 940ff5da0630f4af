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
  * every error path;
  * contexts driven from several threads at once, also under ThreadSanitizer,
    which must report a race planted in a copy of the runtime.
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


def _tsan_build(runtime_dir, exe):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no g++")
    if not os.path.exists(os.path.join(ROCM_INCLUDE, "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not installed")
    # Host code only (g++, no HIP source on this line).
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=thread",
           "-Wall", "-Wextra", "-Werror", "-Wno-unused-parameter",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM_INCLUDE}", f"-I{os.path.join(ROOT, 'include')}",
           f"-I{runtime_dir}", os.path.join(ROOT, "tests", "native", "runtime_host_check.cpp"),
           os.path.join(runtime_dir, "dsm_runtime.cpp"), "-o", exe, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    return subprocess.run([exe, "threads"], capture_output=True, text=True, env=env, timeout=600)


def test_runtime_threads_under_thread_sanitizer(tmp_path):
    r = _tsan_build(CSRC, str(tmp_path / "runtime_threads"))
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "all checks passed" in r.stdout and "ThreadSanitizer" not in r.stderr


def test_thread_sanitizer_sees_a_planted_race(tmp_path):
    """The static-scratch slot released without its lock: the threaded checks
    race on it, and the sanitizer must say so."""
    d = tmp_path / "csrc"
    shutil.copytree(CSRC, d)
    path = d / "dsm_runtime.cpp"
    src = path.read_text()
    lock = ("        std::lock_guard<std::mutex> lock(g_static_mu);\n"
            "        g_static_busy[ctx->static_device] = false;")
    assert src.count(lock) == 1
    path.write_text(src.replace(lock, "        g_static_busy[ctx->static_device] = false;"))
    r = _tsan_build(str(d), str(tmp_path / "runtime_threads_race"))
    assert r.returncode != 0 and "data race" in r.stderr, (r.stdout + r.stderr)[-2000:]
