"""Planted mistakes in the host runtime must fail its CPU harness.

Each case copies the runtime source into a temporary directory, plants one
plausible mistake (in the state machine, the layout, the launch arguments or
the host coefficients), builds tests/native/runtime_host_check.cpp against
the copy with g++ and runs it.  The harness must fail for every mistake.
CPU only, host code only; the real source is untouched.
"""
import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2411_17866_amd", "csrc")
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")

# (original text of dsm_runtime.cpp, planted mistake, what it breaks)
MUTATIONS = [
    ("const dsm::RepLayout sl = from_x ? dsm::single_copy() : ctx->rep;",
     "const dsm::RepLayout sl = ctx->rep;", "stale workers read their own replica"),
    ("const int64_t align = blocked ? dsm::kBlockedTensorAlign : dsm::kTensorAlign;",
     "const int64_t align = dsm::kTensorAlign;", "blocked replicas without the piece alignment"),
    ("    if (blocked) off = round_up(off, block);\n", "",
     "blocked arena not a whole number of blocks"),
    ("        rep = dsm::blocked_copies(problem->n_workers);",
     "        rep = dsm::contiguous_copies(L.arena_elems);",
     "blocked replicas addressed as contiguous copies"),
    ("        ml = dsm::StateLayout{rep, rep, rep};",
     "        ml = dsm::StateLayout{rep, rep, dsm::contiguous_copies(L.arena_elems)};",
     "state-blocked second moments addressed as contiguous copies"),
    ("        rep = dsm::state_blocked_copies(problem->n_workers, nb);",
     "        rep = dsm::state_blocked_copies(problem->n_workers, 4);",
     "state blocks sized for four buffers with the SGD base"),
    ("             (adamw && b->s2_rep != b->x_rep + 3 * gap)))",
     "             (adamw && b->s2_rep != b->x_rep + 2 * gap)))",
     "state-blocked buffer order not checked"),
    ("    a.sl = from_x ? dsm::single_copy() : ctx->rep;", "    a.sl = ctx->rep;",
     "round end after a lazy broadcast reads the stale replicas"),
    ("    ctx->maps = dsm::kMapsByLayout[problem->replica_layout];",
     "    ctx->maps = dsm::kMapsByLayout[0];", "XCD maps of the contiguous layout for every layout"),
    ("    a.map_pass2 = ctx->maps.global;", "    a.map_pass2 = ctx->maps.round_end;",
     "randomized second pass launched with the round-end map"),
    ("ctx->base == DSM_BASE_ADAMW, lc.adam, lc.sgd, ctx->maps.from_x, ctx->stream);",
     "ctx->base == DSM_BASE_ADAMW, lc.adam, lc.sgd, ctx->maps.local, ctx->stream);",
     "step from x launched with the local-step map"),
    ("ctx->buf.x, ctx->buf.x_rep, ctx->rep, ctx->n,\n                                         ctx->maps.copy,",
     "ctx->buf.x, ctx->buf.x_rep, ctx->rep, ctx->n,\n                                         ctx->maps.global,",
     "synchronisation launched with the global-step map"),
    ("        g_static_busy[ctx->static_device] = false;\n", "",
     "a static-scratch context never releases its device"),
    ("        if (need > dsm::kStaticScratchBytes)", "        if (need > 2 * dsm::kStaticScratchBytes)",
     "static scratch limit not enforced"),
    ("        staged.u_scratch = reinterpret_cast<float*>(static_cast<char*>(scratch) + u_off);",
     "        staged.u_scratch = reinterpret_cast<float*>(scratch);",
     "u staging over the static workspace"),
    ("while (b < w0 + nw && ctx->stale[b] == ctx->stale[a]) ++b;",
     "while (b < w0 + nw) ++b;", "runs not split by replica source"),
    ("ctx->stale[i] = broadcast ? 0 : 1;", "ctx->stale[i] = 0;",
     "lazy broadcast leaves replicas marked fresh"),
    ("bool all_stale = worker < 0 && ctx->n > 1;", "bool all_stale = worker < 0;",
     "all-worker step from x taken for n = 1"),
    ("c.off = L->offsets[i] + j;", "c.off = L->offsets[i];", "chunk offset ignores its start"),
    ("sc.bc1 = static_cast<float>(1.0 - beta_power(b1, step));",
     "sc.bc1 = static_cast<float>(1.0 - beta_power(b1, step - 1));", "bias-correction power"),
    ("sc.c2 = static_cast<float>((1.0 - static_cast<double>(hp->beta2)) / gamma);",
     "sc.c2 = static_cast<float>((1.0 - static_cast<double>(hp->beta1)) / gamma);",
     "momentum coefficient uses beta1"),
    ("if (ctx->local_count[i] >= ctx->H)", "if (ctx->local_count[i] > ctx->H)",
     "a local step past H accepted"),
    ("L->bounds_off = L->chunk_bytes;", "L->bounds_off = 0;", "bound words over the chunk table"),
    ("L->chunk0_off = L->bounds_off + round_up(int64_t(p->n_tensors) * 4, 256);",
     "L->chunk0_off = L->bounds_off;", "tensor chunk index over the bounds"),
    ("(*chunk0)[i] = static_cast<int32_t>(k);", "(*chunk0)[i] = static_cast<int32_t>(k + (i > 0));",
     "tensor chunk index off by one"),
    ("round_up(n_chunks * dsm::kSplit * 4, 256)", "round_up(n_chunks * 4, 256)",
     "one piece-maximum word per chunk"),
    ("    if (ctx->n_tensors > 0) {\n        hipError_t e = hipMemcpyAsync(",
     "    if (!ctx->chunks.empty()) {\n        hipError_t e = hipMemcpyAsync(",
     "tensor chunk index not uploaded without chunks"),
    ("ctx->bound.piece_max = reinterpret_cast<uint32_t*>(ws + L.piece_max_off);",
     "ctx->bound.piece_max = reinterpret_cast<uint32_t*>(ws + L.chunk0_off);",
     "piece maxima over the tensor chunk index"),
    ("    if (n_pieces * dsm::kBlockThreads >= (int64_t(1) << 32))",
     "    if (n_pieces * dsm::kBlockThreads >= (int64_t(1) << 40))",
     "streaming diagnostic grid past one dimension"),
    ("    if (kind == DSM_STREAM_READ && n_elems > 0 &&",
     "    if (kind == DSM_STREAM_WRITE && n_elems > 0 &&",
     "streaming read without its word array"),
]


def _run(case, gxx, work):
    original, planted, what = case
    d = os.path.join(work, str(abs(hash(what))))
    shutil.copytree(CSRC, d)
    path = os.path.join(d, "dsm_runtime.cpp")
    src = open(path).read()
    if src.count(original) != 1:
        return what, "original text not found exactly once"
    with open(path, "w") as f:
        f.write(src.replace(original, planted))
    exe = os.path.join(d, "check")
    cmd = [gxx, "-std=c++17", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-static-libasan", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM_INCLUDE}",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{d}",
           os.path.join(ROOT, "tests", "native", "runtime_host_check.cpp"), path, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        return what, "did not build: " + r.stderr[-300:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    return what, None if r.returncode != 0 else "harness passed"


def test_every_planted_runtime_mistake_fails_the_harness():
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no g++")
    if not os.path.exists(os.path.join(ROCM_INCLUDE, "hip", "hip_runtime_api.h")):
        pytest.skip("HIP headers not installed")
    with tempfile.TemporaryDirectory() as work:
        with ThreadPoolExecutor(max_workers=4) as pool:
            results = list(pool.map(lambda c: _run(c, gxx, work), MUTATIONS))
    missed = [f"{what}: {why}" for what, why in results if why is not None]
    assert not missed, "planted runtime mistakes not caught:\n" + "\n".join(missed)
