"""The step calls only enqueue kernels on the context's stream, so a whole
round records into a HIP graph and replays like the eager calls.

A round of Algorithm 1 with the SGD base, the deterministic sign and a
broadcast (H local steps, then the global step) depends on no per-round
scalar: the bias-correction count s and the outer index t only enter AdamW
and the randomized sign.  It also ends with every replica fresh, as it began.
Such a round is captured once and replayed; between replays the same round
runs eagerly on a second set of buffers, with other GPU work and
synchronisations in between, and after every replay both sets must agree bit
for bit.  (Captured scalars are fixed at capture: a round with AdamW's s, the
randomized sign's t or a lazy broadcast is not replayable this way.)  The
randomized sign is also replayed, with the same t on both sides: its two
passes and the bound reduction between them rewrite their workspace words on
every run, so nothing has to be cleared between replays.
"""
import pytest
import torch

from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

NUMEL = [5, 1000, 16385, 40003, 64]
DECAY = [True, False, True, True, False]
N, H = 3, 2
LOCAL = dict(lr=0.05, beta1=0.9)
GLOB = dict(gamma=0.05, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)


def run_round(ctx, mode):
    for k in range(H):
        dsm.dsm_local_step(ctx, -1, k + 1, **LOCAL)
    dsm.dsm_global_step(ctx, 0, broadcast=True, mode=mode, seed=0x5EED, **GLOB)


def bits(t):
    return t.view(torch.int32).clone()


@pytest.mark.parametrize("mode", [dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP],
                         ids=["det", "rand"])
@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("layout", [dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED,
                                    dsm.DSM_REPLICAS_STATE_BLOCKED])
def test_captured_round_replays_like_eager(fused, layout, mode):
    side = torch.cuda.Stream()
    rand = mode != dsm.DSM_SIGN_DET
    eager = A.Arenas(NUMEL, N, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, randomized=rand,
                     replica_layout=layout)
    graph = A.Arenas(NUMEL, N, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, randomized=rand,
                     replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(17)
    eager.x.normal_(0.0, 0.02, generator=gen)
    eager.g_rep.normal_(0.0, 1e-3, generator=gen)
    graph.x.copy_(eager.x)
    graph.g_rep.copy_(eager.g_rep)
    torch.cuda.synchronize()
    eager.init(side)
    graph.init(side)
    side.synchronize()

    def round_(ctx):
        if fused:
            for k in range(H - 1):
                dsm.dsm_local_step(ctx, -1, k + 1, **LOCAL)
            dsm.dsm_round_end(ctx, H, dict(LOCAL), 0, broadcast=True, mode=mode, seed=0x5EED,
                              **GLOB)
        else:
            run_round(ctx, mode)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        round_(graph.ctx)
    torch.cuda.synchronize()
    # Recording ran nothing: both sets still hold the initial state.
    x0 = bits(eager.x)
    assert torch.equal(bits(graph.x), x0)
    scratch = torch.empty(1 << 20, device="cuda")
    for r in range(4):
        with torch.cuda.stream(side):
            round_(eager.ctx)
        side.synchronize()
        scratch.normal_()                       # unrelated eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for name in ("x", "m", "x_rep", "s1_rep"):
            a, b = getattr(eager, name), getattr(graph, name)
            assert torch.equal(bits(a), bits(b)), f"replay {r}: {name} differs from the eager round"
        if rand:
            be = dsm.dsm_read_bounds(eager.ctx, len(NUMEL))
            bg = dsm.dsm_read_bounds(graph.ctx, len(NUMEL))
            assert list(be) == list(bg), f"replay {r}: tensor bounds differ"
        assert not torch.equal(bits(graph.x), x0), "the replayed round did not move the model"
        x0 = bits(graph.x)
    del g
    eager.destroy()
    graph.destroy()
