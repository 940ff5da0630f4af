"""The C ABI from plain C on the GPU: tests/native/c_abi_example.c, built
with gcc against libdsm.so, allocates with hipMalloc and runs a fused lazy
round and a split round with broadcast, then checks the synchronisation
step, the size of the sign step (Eq. (7) with lambda = 0), a round with the
randomized sign of Eq. (10) (its per-tensor bounds against max |u|, its steps
0 or along sign(u)) and error paths; with contiguous replicas and again with
the replicas and their state blocked in one allocation."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "native"))
import c_example_build  # noqa: E402


def test_c_abi_from_plain_c():
    exe = c_example_build.EXE
    if not os.path.exists(exe):
        exe = c_example_build.build()
        if exe is None:
            pytest.skip("no C compiler")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c abi example ok" in r.stdout
