"""The placement probe of arena.Arenas (state-blocked layout): the buffers are
carved at the fastest of several offsets of a larger allocation, timed at
set-up with the problem's own kernels on zeroed buffers.  Where the buffers
sit must not change a single bit of the results, and the probe must leave the
chosen buffers as a fresh allocation would be (zero)."""
import pytest
import torch

from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

NUMEL = [5, 64, 16385, 3000, 0, 40003]
DECAY = [False, True, True, True, True, False]
N, H = 3, 2
GLOB = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1, seed=0x5EED)
LOCAL = {dsm.DSM_BASE_ADAMW: dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
         dsm.DSM_BASE_SGD_MOMENTUM: dict(lr=0.05, beta1=0.9)}
SPAN, STEP = 64 << 20, 16 << 20


def run(ar, base, gen_seed):
    gen = torch.Generator(device="cuda").manual_seed(gen_seed)
    ar.x.normal_(0.0, 0.02, generator=gen)
    ar.init()
    s = 0
    for t, (mode, fused) in enumerate([(dsm.DSM_SIGN_RAND_FLIP, True), (dsm.DSM_SIGN_DET, False)]):
        for k in range(H):
            ar.g_rep.normal_(0.0, 1e-3, generator=gen)
            s += 1
            if fused and k == H - 1:
                dsm.dsm_round_end(ar.ctx, s, LOCAL[base], t, mode=mode, broadcast=False, **GLOB)
            else:
                dsm.dsm_local_step(ar.ctx, -1, s, **LOCAL[base])
        if not fused:
            dsm.dsm_global_step(ar.ctx, t, mode=mode, broadcast=True, **GLOB)
    torch.cuda.synchronize()
    names = ("x", "m", "x_rep", "s1_rep") + (("s2_rep",) if base == dsm.DSM_BASE_ADAMW else ())
    return {k: getattr(ar, k).contiguous().view(torch.int32).clone() for k in names}


@pytest.mark.parametrize("base", [dsm.DSM_BASE_ADAMW, dsm.DSM_BASE_SGD_MOMENTUM])
def test_probed_placement_gives_the_same_bits(base):
    ref = A.Arenas(NUMEL, N, H, base, decay=DECAY, randomized=True,
                   replica_layout=dsm.DSM_REPLICAS_STATE_BLOCKED)
    assert ref.placement is None
    got = A.Arenas(NUMEL, N, H, base, decay=DECAY, randomized=True,
                   replica_layout=dsm.DSM_REPLICAS_STATE_BLOCKED,
                   placement_span=SPAN, placement_step=STEP)
    p = got.placement
    assert p["candidates"] == SPAN // STEP + 1
    assert p["offset_bytes"] % (2 << 20) == 0 and 0 <= p["offset_bytes"] <= SPAN
    assert p["best_ms"] <= p["worst_ms"]
    # The chosen buffers start zeroed, as a fresh allocation's are.
    for name in ("x", "m", "u", "x_rep_flat"):
        assert not getattr(got, name).any(), f"{name} not zeroed after the probe"
    want = run(ref, base, 7)
    have = run(got, base, 7)
    ref.destroy()
    got.destroy()
    for k in want:
        assert torch.equal(want[k], have[k]), f"{k} differs with the probed placement"
