"""Two contexts at once: each on its own stream, driven from its own host
thread, give bit for bit the results they give one after the other.

A context keeps all of its state in its own host object and the caller's
buffers (the error text of a failed call is per thread), so contexts do not
interact.  ctypes releases the interpreter lock during each call, so the two
threads are inside the library at the same time.  The first context is also
run from dsm_init_static, whose workspace is the library's static scratch,
beside an ordinary one.
"""
import threading

import pytest
import torch

from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

PROBLEMS = [
    dict(numel=[5, 1000, 16385, 40003], n=3, H=2, base=dsm.DSM_BASE_ADAMW,
         local=dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)),
    dict(numel=[64, 70001, 3], n=4, H=3, base=dsm.DSM_BASE_SGD_MOMENTUM,
         local=dict(lr=0.05, beta1=0.9)),
]
GLOB = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1, seed=0x1234ABCD)
ROUNDS = 4


def setup(spec, seed):
    ar = A.Arenas(spec["numel"], spec["n"], spec["H"], spec["base"], randomized=True)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    ar.x.normal_(0.0, 0.02, generator=gen)
    grads = [torch.empty_like(ar.g_rep).normal_(0.0, 1e-3, generator=gen)
             for _ in range(ROUNDS * spec["H"])]
    torch.cuda.synchronize()
    return ar, grads


def drive(ar, spec, grads, stream, static=False):
    """ROUNDS rounds: fused lazy and split rounds, both signs, on `stream`."""
    with torch.cuda.stream(stream):
        if static:
            bufs = ar.buffers(stream)
            bufs.workspace, bufs.workspace_bytes, bufs.u_scratch = None, 0, None
            ar.ctx = dsm.dsm_init_static(ar.problem, bufs)
        else:
            ar.init(stream)
        H = spec["H"]
        for t in range(ROUNDS):
            mode = (dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP, dsm.DSM_SIGN_RAND_ZERO)[t % 3]
            for k in range(H):
                ar.g_rep.copy_(grads[t * H + k])
                s = t * H + k + 1
                if t % 2 == 0 and k == H - 1:
                    dsm.dsm_round_end(ar.ctx, s, spec["local"], t, mode=mode, broadcast=False, **GLOB)
                else:
                    dsm.dsm_local_step(ar.ctx, -1, s, **spec["local"])
            if t % 2 == 1:
                dsm.dsm_global_step(ar.ctx, t, mode=mode, broadcast=True, **GLOB)
        dsm.dsm_sync(ar.ctx)
    stream.synchronize()


def state(ar):
    return {name: getattr(ar, name).view(torch.int32).clone()
            for name in ("x", "m", "x_rep", "s1_rep")}


@pytest.mark.parametrize("static_first", [False, True], ids=["init", "init_static"])
def test_two_contexts_on_two_streams_from_two_threads(static_first):
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    static = [static_first, False]
    # One after the other.
    want = []
    for i, spec in enumerate(PROBLEMS):
        ar, grads = setup(spec, 100 + i)
        drive(ar, spec, grads, streams[i], static[i])
        want.append(state(ar))
        ar.destroy()
    # At the same time, from two threads.
    runs = [setup(spec, 100 + i) for i, spec in enumerate(PROBLEMS)]
    errors = []

    def work(i):
        try:
            drive(runs[i][0], PROBLEMS[i], runs[i][1], streams[i], static[i])
        except Exception as e:          # reported below, in the main thread
            errors.append(repr(e))
    threads = [threading.Thread(target=work, args=(i,)) for i in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    assert not any(th.is_alive() for th in threads)
    torch.cuda.synchronize()
    for i in range(2):
        got = state(runs[i][0])
        for name in want[i]:
            assert torch.equal(got[name], want[i][name]), f"context {i}: {name} differs"
        runs[i][0].destroy()

