"""dsm_init_static, the entry point that allocates nothing, against dsm_init.

Three problems in a row, each smaller than the one before, so the second context starts from
the static scratch the first one left behind.  Each is run twice from the same
seeded start: once on a context from dsm_init (caller workspace and u
staging) and once on a context from dsm_init_static, whose buffers carry no
workspace and no u staging at all.  Three rounds each: split deterministic
with broadcast, split randomized (Eq. (9)) with broadcast, fused randomized
(Eq. (10)) with the lazy broadcast.  Every state buffer and every bound must
be bit-identical.  Also: a second static context on the device is refused
while the first is alive, and a problem beyond the scratch is refused.
"""
import numpy as np
import pytest
import torch

from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

CASES = [  # (numel, n, H, base, layout): the second one smaller
    ([16385, 40003, 5, 100000, 0, 63], 3, 2, dsm.DSM_BASE_ADAMW, dsm.DSM_REPLICAS_BLOCKED),
    ([40000, 1000], 2, 2, dsm.DSM_BASE_ADAMW, dsm.DSM_REPLICAS_STATE_BLOCKED),
    ([1000, 7], 2, 1, dsm.DSM_BASE_SGD_MOMENTUM, dsm.DSM_REPLICAS_CONTIGUOUS),
]
LOCAL = {dsm.DSM_BASE_ADAMW: dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
         dsm.DSM_BASE_SGD_MOMENTUM: dict(lr=0.05, beta1=0.9)}
GLOB = dict(eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)
ROUNDS = [(dsm.DSM_SIGN_DET, False, True), (dsm.DSM_SIGN_RAND_FLIP, False, True),
          (dsm.DSM_SIGN_RAND_ZERO, True, False)]   # (mode, fused, broadcast)


def _state(ar):
    torch.cuda.synchronize()
    out = {"x": ar.x, "m": ar.m, "x_rep": ar.replicas(), "s1": ar.workers("s1_rep")}
    if ar.s2_rep is not None:
        out["s2"] = ar.workers("s2_rep")
    return {k: v.detach().cpu().numpy().view(np.uint32).copy() for k, v in out.items()}


def _run(case, static):
    numel, n, H, base, layout = case
    local = LOCAL[base]
    ar = A.Arenas(numel, n, H, base, randomized=True, replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(2024)
    ar.x.normal_(0.0, 0.02, generator=gen)
    bufs = ar.buffers()
    if static:
        bufs.workspace, bufs.workspace_bytes, bufs.u_scratch = None, 0, None
        ar.ctx = dsm.dsm_init_static(ar.problem, bufs)
        # While it is alive, the device's scratch is taken.
        with pytest.raises(dsm.DsmError) as e:
            dsm.dsm_init_static(ar.problem, bufs)
        assert e.value.status == dsm.DSM_ERR_STATE
    else:
        ar.ctx = dsm.dsm_init(ar.problem, bufs)
    states, bounds = [], []
    s = 0
    for t, (mode, fused, broadcast) in enumerate(ROUNDS):
        for k in range(H):
            ar.g_rep.normal_(0.0, 1e-3, generator=gen)
            s += 1
            if fused and k == H - 1:
                dsm.dsm_round_end(ar.ctx, s, local, t, gamma=local["lr"], mode=mode, seed=99,
                                  broadcast=broadcast, **GLOB)
            else:
                dsm.dsm_local_step(ar.ctx, -1, s, **local)
        if not fused:
            dsm.dsm_global_step(ar.ctx, t, gamma=local["lr"], mode=mode, seed=99,
                                broadcast=broadcast, **GLOB)
        states.append(_state(ar))
        bounds.append(dsm.dsm_read_bounds(ar.ctx, len(numel)).view(np.uint32).copy()
                      if mode != dsm.DSM_SIGN_DET else None)
    ar.destroy()
    return states, bounds


def test_static_scratch_context_matches_dsm_init():
    for case in CASES:
        ref_states, ref_bounds = _run(case, static=False)
        got_states, got_bounds = _run(case, static=True)
        for t, (a, b) in enumerate(zip(ref_states, got_states)):
            for key in a:
                assert np.array_equal(a[key], b[key]), (case[0], t, key)
        for t, (a, b) in enumerate(zip(ref_bounds, got_bounds)):
            if a is not None:
                assert np.array_equal(a, b), (case[0], t, "bounds")


def test_static_scratch_refuses_a_problem_beyond_it():
    numel = [(64 << 20) // 4 + 1]
    prob = dsm.make_problem(numel, 1, 1, dsm.DSM_BASE_SGD_MOMENTUM)
    with pytest.raises(dsm.DsmError) as e:     # refused before any buffer is looked at
        dsm.dsm_init_static(prob, dsm.dsm_buffers())
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG
    assert "static scratch" in e.value.message


@pytest.mark.parametrize("mode", [dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP], ids=["det", "rand"])
def test_static_context_round_replays_from_a_graph(mode):
    """The callers it is for include code under graph capture: a round of a
    static-scratch context (SGD base, broadcast, the same t every round)
    records into a HIP graph and each replay matches an eager dsm_init round."""
    numel, n, H = [5, 16385, 40003, 64], 3, 2
    local = LOCAL[dsm.DSM_BASE_SGD_MOMENTUM]
    side = torch.cuda.Stream()
    eager = A.Arenas(numel, n, H, dsm.DSM_BASE_SGD_MOMENTUM, randomized=True)
    graph = A.Arenas(numel, n, H, dsm.DSM_BASE_SGD_MOMENTUM, randomized=True)
    gen = torch.Generator(device="cuda").manual_seed(5)
    eager.x.normal_(0.0, 0.02, generator=gen)
    eager.g_rep.normal_(0.0, 1e-3, generator=gen)
    graph.x.copy_(eager.x)
    graph.g_rep.copy_(eager.g_rep)
    torch.cuda.synchronize()
    eager.ctx = dsm.dsm_init(eager.problem, eager.buffers(side))
    bufs = graph.buffers(side)
    bufs.workspace, bufs.workspace_bytes, bufs.u_scratch = None, 0, None
    graph.ctx = dsm.dsm_init_static(graph.problem, bufs)
    side.synchronize()

    def round_(ctx):
        for k in range(H):
            dsm.dsm_local_step(ctx, -1, k + 1, **local)
        dsm.dsm_global_step(ctx, 0, gamma=local["lr"], mode=mode, seed=7, broadcast=True, **GLOB)

    try:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            round_(graph.ctx)
        torch.cuda.synchronize()
        for r in range(3):
            with torch.cuda.stream(side):
                round_(eager.ctx)
            side.synchronize()
            g.replay()
            torch.cuda.synchronize()
            a, b = _state(eager), _state(graph)
            for key in a:
                assert np.array_equal(a[key], b[key]), (r, key)
        del g
    finally:
        graph.destroy()
        eager.destroy()
