"""Host-side tests of the C ABI (no GPU needed): the library loads and exports
every entry point include/dsm.h declares; dsm_layout; and every argument
error detected on the host before any device work."""
import ctypes
import os
import re
import threading

import numpy as np
import pytest

from paper_2411_17866_amd import dsm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _no_gpu():
    try:
        import torch
        return not torch.cuda.is_available()
    except Exception:
        return True


needs_no_gpu = pytest.mark.skipif(not _no_gpu(), reason="uses fake device pointers; CPU host only")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(dsm.LIBPATH):
        from paper_2411_17866_amd import build
        build.build()
    return dsm.load_library()


def test_exports_every_declared_entry_point(lib):
    header = open(os.path.join(ROOT, "include", "dsm.h")).read()
    declared = set(re.findall(r"^DSM_API [^(]*?\b(dsm_\w+)\(", header, flags=re.M))
    assert declared == set(dsm.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name
    # Nothing else leaks out of the library's dynamic symbol table.
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", dsm.LIBPATH], capture_output=True,
                         text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.split()[-2] in "TW"}
    assert {s for s in exported if s.startswith("dsm_")} == declared


def test_layout_offsets_aligned_and_packed(lib):
    numel = [1, 3, 64, 65, 0, 16384, 16385, 100000]
    prob = dsm.make_problem(numel, 4, 2, dsm.DSM_BASE_ADAMW)
    arena, offs, ws = dsm.dsm_layout(prob)
    expect, o = [], 0
    for n in numel:
        expect.append(o)
        o += -(-n // 64) * 64
    assert list(offs) == expect
    assert arena == o
    # Chunk table (32 B per chunk), bound words (4 B per tensor), first chunk
    # of each tensor (4 B per tensor, plus one), one piece-maximum word per
    # 1024-element work-group piece; each part rounded up to 256 B.
    n_chunks = sum(-(-n // 16384) for n in numel)
    up = lambda b: -(-b // 256) * 256
    assert ws == (up(n_chunks * 32) + up(len(numel) * 4) + up((len(numel) + 1) * 4)
                  + up(n_chunks * 16 * 4))


def test_layout_empty_problem(lib):
    prob = dsm.make_problem([], 1, 1, dsm.DSM_BASE_SGD_MOMENTUM)
    arena, offs, ws = dsm.dsm_layout(prob)
    assert arena == 0 and len(offs) == 0 and ws == 0


@pytest.mark.parametrize("kw,msg", [
    (dict(numel=[4], n=0), "n_workers"),
    (dict(numel=[4], n=65), "n_workers"),
    (dict(numel=[4], H=0), "local_steps"),
    (dict(numel=[-1]), "numel"),
    (dict(numel=[1 << 34]), "numel"),
    (dict(numel=[4], base=7), "base"),
])
def test_layout_rejects_invalid_problems(lib, kw, msg):
    prob = dsm.make_problem(kw.get("numel"), kw.get("n", 2), kw.get("H", 2), kw.get("base", 0))
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_layout(prob)
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG
    assert msg in e.value.message
    assert msg in dsm.dsm_last_error(None)


def _fake_buffers(arena, n, ws, misalign=None, null=None, ws_bytes=None, adamw=True):
    base = 1 << 40
    names = ["x", "m", "x_rep", "g_rep", "s1_rep", "s2_rep", "u_scratch", "workspace"]
    ptrs = {}
    for i, name in enumerate(names):
        ptrs[name] = base + i * (1 << 34)
    if not adamw:
        ptrs["s2_rep"] = None
    if misalign:
        ptrs[misalign] += 4
    if null:
        ptrs[null] = None
    return dsm.dsm_buffers(ptrs["x"], ptrs["m"], ptrs["x_rep"], ptrs["g_rep"], ptrs["s1_rep"],
                           ptrs["s2_rep"], ptrs["u_scratch"], ptrs["workspace"],
                           ws if ws_bytes is None else ws_bytes, None, None)


@needs_no_gpu
@pytest.mark.parametrize("case", ["misalign_x", "null_m", "null_s2", "small_ws", "misalign_ws"])
def test_init_rejects_bad_buffers_on_host(lib, case):
    prob = dsm.make_problem([1000, 7], 2, 3, dsm.DSM_BASE_ADAMW)
    arena, _, ws = dsm.dsm_layout(prob)
    kw = {"misalign_x": dict(misalign="x"), "null_m": dict(null="m"),
          "null_s2": dict(null="s2_rep"), "small_ws": dict(ws_bytes=ws - 1),
          "misalign_ws": dict(misalign="workspace")}[case]
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_init(prob, _fake_buffers(arena, 2, ws, **kw))
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG


@needs_no_gpu
def test_init_without_device_reports_hip_error(lib):
    """Valid arguments on a host with no GPU: DSM_ERR_HIP, nothing dereferenced."""
    prob = dsm.make_problem([1000, 7], 2, 3, dsm.DSM_BASE_SGD_MOMENTUM)
    arena, _, ws = dsm.dsm_layout(prob)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_init(prob, _fake_buffers(arena, 2, ws, adamw=False))
    assert e.value.status == dsm.DSM_ERR_HIP
    assert "no HIP device" in e.value.message


def test_null_context_is_an_argument_error(lib):
    for call in (lambda: dsm.dsm_local_step(None, -1, 1, 1e-3, 0.9, 0.95, 1e-8, 0.0),
                 lambda: dsm.dsm_global_step(None, 0, 1e-3, 1.0, 0.9, 0.99, 0.1),
                 lambda: dsm.dsm_sync(None)):
        with pytest.raises(dsm.DsmError) as e:
            call()
        assert e.value.status == dsm.DSM_ERR_INVALID_ARG
    assert lib.dsm_read_bounds(None, None, 0) == dsm.DSM_ERR_INVALID_ARG
    assert lib.dsm_destroy(None) == dsm.DSM_OK


@needs_no_gpu
@pytest.mark.parametrize("args", [
    (0, 0, 0, 0, 4, None),            # NULL output
    (0, 0, 0, -1, 4, 1 << 40),        # negative q0
    (0, 0, 0, (1 << 32) - 2, 4, 1 << 40),  # counter overflow
    (0, 0, 1 << 32, 0, 4, 1 << 40),   # t out of range
    (0, 0, 0, 0, 4, (1 << 40) + 2),   # misaligned output
])
def test_test_philox_rejects_bad_arguments(lib, args):
    seed, tensor, t, q0, count, out = args
    st = lib.dsm_test_philox(seed, tensor, t, q0, count, out, None)
    assert st == dsm.DSM_ERR_INVALID_ARG


@needs_no_gpu
@pytest.mark.parametrize("args", [
    (2, 1 << 40, 1024, 1 << 40),          # unknown kind
    (1, 1 << 40, 1000, None),             # not whole pieces
    (1, 1 << 40, -1024, None),            # negative size
    (1, 1 << 40, (1 << 24) * 1024, None),  # beyond one grid dimension
    (0, 1 << 40, 1024, None),             # read without the word array
    (1, (1 << 40) + 16, 1024, None),      # misaligned buffer
    (1, None, 1024, None),                # NULL buffer
])
def test_test_stream_rejects_bad_arguments(lib, args):
    kind, buf, n, words = args
    assert lib.dsm_test_stream(kind, buf, n, words, 0, None) == dsm.DSM_ERR_INVALID_ARG


def test_struct_layouts_match_header(lib):
    """ctypes mirrors of the header structs have the C sizes and offsets."""
    assert ctypes.sizeof(dsm.dsm_problem) == 40
    assert dsm.dsm_problem.numel.offset == 16
    assert dsm.dsm_problem.replica_layout.offset == 32
    assert ctypes.sizeof(dsm.dsm_buffers) == 88
    assert dsm.dsm_buffers.stream.offset == 72
    assert ctypes.sizeof(dsm.dsm_local_hparams) == 20
    assert ctypes.sizeof(dsm.dsm_global_hparams) == 40
    assert dsm.dsm_global_hparams.seed.offset == 24


def test_header_compiles_as_c_and_struct_sizes_agree(tmp_path):
    """The public header is plain C; its struct sizes match the ctypes mirror."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "t.c"
    src.write_text('#include "dsm.h"\n#include <stdio.h>\n#include <stddef.h>\n'
                   'int main(void){printf("%zu %zu %zu %zu %zu %zu %zu\\n", sizeof(dsm_problem),'
                   ' sizeof(dsm_buffers), sizeof(dsm_local_hparams), sizeof(dsm_global_hparams),'
                   ' offsetof(dsm_buffers, stream), offsetof(dsm_global_hparams, seed),'
                   ' offsetof(dsm_problem, replica_layout));'
                   'return 0;}\n')
    exe = tmp_path / "t"
    subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()
    assert [int(v) for v in out] == [40, 88, 20, 40, 72, 24, 32]


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(dsm, "_lib", None)
    with pytest.raises(RuntimeError, match="not found"):
        dsm.load_library(str(tmp_path / "missing.so"))


def test_error_text_is_per_thread():
    """A failing call in one thread does not change the error text another
    thread reads for its own failure (no context: the thread's last error).
    Host only."""
    out = {}

    def fail(tag, n_workers):
        prob = dsm.make_problem([8], n_workers, 1, dsm.DSM_BASE_ADAMW)
        with pytest.raises(dsm.DsmError):
            dsm.dsm_layout(prob)
        out[tag] = dsm.dsm_last_error()
    ths = [threading.Thread(target=fail, args=("zero", 0)),
           threading.Thread(target=fail, args=("many", 65))]
    for th in ths:
        th.start()
    for th in ths:
        th.join(timeout=60)
    assert "got 0" in out["zero"] and "got 65" in out["many"]
