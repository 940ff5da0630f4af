"""The fused round boundary against the unfused calls and the oracle.

dsm_round_end (local step H of every worker fused with the global step) and
the lazy broadcast (a global step with broadcast = 0; each worker's next
local step reads x) must give results bit-identical to H x dsm_local_step +
dsm_global_step(broadcast = 1), and to the oracle's rounds of Algorithm 1.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

NUMEL = [5, 64, 16385, 40003, 1000]
DECAY = [False, True, True, True, False]
ADAM = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
SGD = dict(lr=0.05, beta1=0.9)
GLOB = dict(eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().copy()


def tensors(ar, flat):
    h = host(flat)
    return [h[o:o + k].copy() for o, k in zip(ar.offsets, ar.numel)]


def _grads(ar, t, k):
    gen = torch.Generator(device="cuda").manual_seed(1000 * t + k)
    ar.g_rep.normal_(0.0, 0.01, generator=gen)


LAYOUTS = [dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED, dsm.DSM_REPLICAS_STATE_BLOCKED]


def run(base, mode, broadcast, n, H, fused, rounds=3, record_grads=False,
        layout=dsm.DSM_REPLICAS_CONTIGUOUS):
    local = ADAM if base == dsm.DSM_BASE_ADAMW else SGD
    ar = A.Arenas(NUMEL, n, H, base, decay=DECAY, randomized=mode != dsm.DSM_SIGN_DET,
                  replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(77)
    ar.x.normal_(0.0, 0.02, generator=gen)
    ar.init()
    grads = {}
    for t in range(rounds):
        for k in range(H):
            _grads(ar, t, k)
            if record_grads:
                for i in range(n):
                    grads[(t, i, k)] = tensors(ar, ar.worker("g_rep", i))
            s = t * H + k + 1
            if fused and k == H - 1:
                dsm.dsm_round_end(ar.ctx, s, local, t, gamma=local["lr"], mode=mode, seed=9,
                                  broadcast=broadcast, **GLOB)
            else:
                dsm.dsm_local_step(ar.ctx, -1, s, **local)
        if not fused:
            dsm.dsm_global_step(ar.ctx, t, gamma=local["lr"], mode=mode, seed=9,
                                broadcast=broadcast, **GLOB)
    out = {"x": host(ar.x), "m": host(ar.m), "s1": host(ar.workers("s1_rep"))}
    if ar.s2_rep is not None:
        out["s2"] = host(ar.workers("s2_rep"))
    if broadcast:
        out["x_rep"] = host(ar.replicas())
    if mode != dsm.DSM_SIGN_DET:
        out["B"] = dsm.dsm_read_bounds(ar.ctx, len(NUMEL))
        out["u"] = host(ar.u)
    offsets = list(ar.offsets)
    ar.destroy()
    return out, grads, offsets


def _mask(offsets, arena):
    mask = np.zeros(arena, dtype=bool)
    for o, k in zip(offsets, NUMEL):
        mask[o:o + k] = True
    return mask


@pytest.mark.parametrize("base", [dsm.DSM_BASE_ADAMW, dsm.DSM_BASE_SGD_MOMENTUM])
@pytest.mark.parametrize("mode", [dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP, dsm.DSM_SIGN_RAND_ZERO])
@pytest.mark.parametrize("broadcast", [True, False])
@pytest.mark.parametrize("n,H", [(4, 3), (3, 1), (1, 2)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_fused_round_end_bit_identical_to_unfused(base, mode, broadcast, n, H, layout):
    ref, _, offsets = run(base, mode, broadcast=True, n=n, H=H, fused=False, layout=layout)
    got, _, _ = run(base, mode, broadcast=broadcast, n=n, H=H, fused=True, layout=layout)
    keep = _mask(offsets, ref["x"].size)
    for key in ("x", "m", "s1", "s2", "u"):
        if key in got:
            a, b = ref[key], got[key]
            sel = keep if a.ndim == 1 else np.broadcast_to(keep, a.shape)
            assert np.array_equal(a[sel].view(np.uint32), b[sel].view(np.uint32)), key
    if "B" in got:
        assert np.array_equal(ref["B"].view(np.uint32), got["B"].view(np.uint32))
    if broadcast:
        sel = np.broadcast_to(keep, ref["x_rep"].shape)
        assert np.array_equal(ref["x_rep"][sel].view(np.uint32), got["x_rep"][sel].view(np.uint32))


@pytest.mark.parametrize("base", [dsm.DSM_BASE_ADAMW, dsm.DSM_BASE_SGD_MOMENTUM])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_fused_lazy_rounds_match_oracle(base, layout):
    """Three fused rounds with the lazy broadcast against the oracle's rounds
    (fp32), free-running: x, m and the base state bit-identical."""
    n, H = 3, 2
    got, grads, offsets = run(base, dsm.DSM_SIGN_DET, broadcast=False, n=n, H=H, fused=True,
                              record_grads=True, layout=layout)
    local = ADAM if base == dsm.DSM_BASE_ADAMW else SGD
    ar = A.Arenas(NUMEL, n, H, base, decay=DECAY, randomized=False, replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(77)
    ar.x.normal_(0.0, 0.02, generator=gen)
    x0 = tensors(ar, ar.x)
    ar.destroy()
    st = O.init_state(x0, n, "adamw" if base == dsm.DSM_BASE_ADAMW else "sgd")
    for t in range(3):
        O.communication_round(st, lambda i, k: grads[(t, i, k)], t, H=H, local=local,
                              glob=dict(GLOB, mode=O.SIGN_DET, seed=0), decay=DECAY, prec="fp32")
    for p, (o, k) in enumerate(zip(offsets, NUMEL)):
        assert np.array_equal(got["x"][o:o + k].view(np.uint32), st["x"][p].view(np.uint32))
        assert np.array_equal(got["m"][o:o + k].view(np.uint32), st["m"][p].view(np.uint32))
        for i in range(n):
            assert np.array_equal(got["s1"][i, o:o + k], st["s1"][i][p])


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mixed_stale_and_fresh_workers(layout):
    """After a global step without broadcast, a single worker's local step
    reads x; a following all-worker step mixes stale and fresh replicas.
    SGD base (no bias-correction count), one gradient per worker per round."""
    n, H = 3, 2
    ar = A.Arenas(NUMEL, n, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, randomized=False,
                  replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(5)
    ar.x.normal_(0.0, 0.02, generator=gen)
    ar.init()
    st = O.init_state(tensors(ar, ar.x), n, "sgd")
    for t in range(2):
        ar.g_rep.normal_(0.0, 0.01, generator=gen)
        g = [tensors(ar, ar.worker("g_rep", i)) for i in range(n)]
        if t == 0:
            dsm.dsm_local_step(ar.ctx, -1, 1, **SGD)
            dsm.dsm_local_step(ar.ctx, -1, 2, **SGD)
        else:
            dsm.dsm_local_step(ar.ctx, 1, 1, **SGD)     # worker 1 reads x
            dsm.dsm_local_step(ar.ctx, -1, 1, **SGD)    # 0, 2 read x; 1 its replica
            dsm.dsm_local_step(ar.ctx, 0, 2, **SGD)
            dsm.dsm_local_step(ar.ctx, 2, 2, **SGD)
        dsm.dsm_global_step(ar.ctx, t, gamma=SGD["lr"], broadcast=False, **GLOB)
        O.communication_round(st, lambda i, k: g[i], t, H=H, local=SGD,
                              glob=dict(GLOB, mode=O.SIGN_DET, seed=0), decay=DECAY, prec="fp32")
        gx = tensors(ar, ar.x)
        for p in range(len(NUMEL)):
            assert np.array_equal(gx[p].view(np.uint32), st["x"][p].view(np.uint32)), (t, p)
    ar.destroy()


def test_round_end_state_errors():
    ar = A.Arenas([100], 2, 3, dsm.DSM_BASE_ADAMW, randomized=False)
    ar.init()
    with pytest.raises(dsm.DsmError) as e:   # needs H - 1 = 2 local steps first
        dsm.dsm_round_end(ar.ctx, 1, ADAM, 0, gamma=1e-3, **GLOB)
    assert e.value.status == dsm.DSM_ERR_STATE
    dsm.dsm_local_step(ar.ctx, -1, 1, **ADAM)
    dsm.dsm_local_step(ar.ctx, -1, 2, **ADAM)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_round_end(ar.ctx, 3, ADAM, 0, gamma=1e-3, mode=dsm.DSM_SIGN_RAND_FLIP, **GLOB)
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG       # no u_scratch
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_round_end(ar.ctx, 0, ADAM, 0, gamma=1e-3, **GLOB)
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG       # step 0
    dsm.dsm_round_end(ar.ctx, 3, ADAM, 0, gamma=1e-3, **GLOB)
    ar.destroy()


@pytest.mark.parametrize("base", [dsm.DSM_BASE_ADAMW, dsm.DSM_BASE_SGD_MOMENTUM])
@pytest.mark.parametrize("n", [2, 3, 4, 5, 8])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_all_worker_step_from_x_equals_per_worker_steps(base, n, layout):
    """After a global step without broadcast every replica is stale.  A local
    step of all workers then reads x once in one launch; it must equal n
    single-worker steps (each reading x) bit for bit, and so must the rest of
    the round."""
    local = ADAM if base == dsm.DSM_BASE_ADAMW else SGD
    H = 2
    outs = []
    for per_worker in (False, True):
        ar = A.Arenas(NUMEL, n, H, base, decay=DECAY, randomized=False, replica_layout=layout)
        gen = torch.Generator(device="cuda").manual_seed(5 + n)
        ar.x.normal_(0.0, 0.02, generator=gen)
        ar.init()
        for k in range(H):
            _grads(ar, 0, k)
            dsm.dsm_local_step(ar.ctx, -1, k + 1, **local)
        dsm.dsm_global_step(ar.ctx, 0, gamma=local["lr"], broadcast=False, **GLOB)
        _grads(ar, 1, 0)
        if per_worker:
            for i in range(n):
                dsm.dsm_local_step(ar.ctx, i, H + 1, **local)
        else:
            dsm.dsm_local_step(ar.ctx, -1, H + 1, **local)
        first = {"x_rep": host(ar.replicas()), "s1": host(ar.workers("s1_rep"))}
        if ar.s2_rep is not None:
            first["s2"] = host(ar.workers("s2_rep"))
        _grads(ar, 1, 1)
        dsm.dsm_local_step(ar.ctx, -1, H + 2, **local)
        dsm.dsm_global_step(ar.ctx, 1, gamma=local["lr"], broadcast=True, **GLOB)
        after = {"x": host(ar.x), "m": host(ar.m), "x_rep_end": host(ar.replicas())}
        mask = _mask(list(ar.offsets), ar.x.numel())
        ar.destroy()
        outs.append((first, after, mask))
    (fa, aa, mask), (fb, ab, _) = outs
    for key in fa:
        for i in range(n):
            a, b = fa[key][i][mask], fb[key][i][mask]
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), (key, i)
    for key in ("x", "m"):
        assert np.array_equal(aa[key][mask].view(np.uint32), ab[key][mask].view(np.uint32)), key
    for i in range(n):
        assert np.array_equal(aa["x_rep_end"][i][mask].view(np.uint32),
                              ab["x_rep_end"][i][mask].view(np.uint32))
