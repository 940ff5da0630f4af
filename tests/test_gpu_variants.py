"""GPU global-step variants (Lookahead, signed SlowMo, Global AdamW) against
the oracle, through the C ABI, on ragged multi-chunk tensors."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

from parity import U32, rel_check, rms

pytestmark = pytest.mark.gpu

RAGGED = [1, 3, 5, 64, 65, 0, 1000, 16383, 16385, 40003]
DECAY = [i % 3 != 1 for i in range(len(RAGGED))]
SGD = dict(lr=0.05, beta1=0.5)
GLOB = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)
ADAMW_GLOB = dict(gamma=1e-3, eta=1e-3, beta1=0.9, beta2=0.95, lam=0.1, eps=1e-8)
RULES = {dsm.DSM_RULE_LOOKAHEAD: O.RULE_LOOKAHEAD, dsm.DSM_RULE_SIGNED_SLOWMO: O.RULE_SIGNED_SLOWMO,
         dsm.DSM_RULE_GLOBAL_ADAMW: O.RULE_GLOBAL_ADAMW}


def tensors(ar, flat):
    torch.cuda.synchronize()
    h = flat.detach().cpu().numpy()
    return [h[o:o + k].copy() for o, k in zip(ar.offsets, ar.numel)]


def _run_variant(rule, n, broadcast, rounds, seed, layout=dsm.DSM_REPLICAS_CONTIGUOUS):
    adamw = rule == dsm.DSM_RULE_GLOBAL_ADAMW
    hp = ADAMW_GLOB if adamw else GLOB
    H = 2
    ar = A.Arenas(RAGGED, n, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, randomized=False,
                  global_adamw=adamw, replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    ar.x.normal_(0.0, 0.02, generator=gen)
    ar.init()
    if not adamw:
        ar.m.normal_(0.0, 1.0, generator=gen)
    nonbit = 0
    for t in range(rounds):
        for k in range(H):
            ar.g_rep.normal_(0.0, 1e-3, generator=gen)
            dsm.dsm_local_step(ar.ctx, -1, 1, **SGD)
        x0, m0 = tensors(ar, ar.x), tensors(ar, ar.m)
        v0 = tensors(ar, ar.v) if adamw else None
        reps = [tensors(ar, ar.replica(i)) for i in range(n)]
        dsm.dsm_global_step(ar.ctx, t, rule=rule, broadcast=broadcast, **hp)
        gx, gm = tensors(ar, ar.x), tensors(ar, ar.m)
        okw = dict(hp, decay=DECAY, t=t, rule=RULES[rule])
        if adamw:
            okw["v"] = v0
        o32 = O.global_step(x0, m0, reps, prec="fp32", **okw)
        o64 = O.global_step(x0, m0, reps, prec="fp64", **okw)
        for p in range(len(RAGGED)):
            nonbit += rel_check(gx[p], o32["x"][p], f"rule {rule} t {t} x tensor {p}")
            nonbit += rel_check(gm[p], o32["m"][p], f"rule {rule} t {t} m tensor {p}")
            if adamw:
                nonbit += rel_check(tensors(ar, ar.v)[p], o32["v"][p], f"v tensor {p}")
            # fp64 reference: the fp32 path stays within a small multiple of
            # u of the magnitudes of the terms of the update (|S| <= 1 and the
            # AdamW ratio is O(1), hence the 1); sign decisions of signed
            # SlowMo may differ only where the averaged difference is tiny.
            ok = np.ones(RAGGED[p], dtype=bool)
            if rule == dsm.DSM_RULE_SIGNED_SLOWMO:
                flip = np.sign(o32["delta"][p]) != np.sign(o64["delta"][p])
                if flip.any():
                    assert np.all(np.abs(o64["delta"][p][flip]) < 1e-6 * rms(o64["delta"][p]))
                ok &= ~flip
            err = np.abs(gx[p].astype(np.float64) - o64["x"][p])
            bound = 64 * U32 * (np.abs(o64["x"][p]) + np.abs(x0[p]) +
                                O.f32(hp["eta"]) * (O.f32(hp["gamma"]) if not adamw else 1.0) *
                                (np.abs(o64["u"][p]) + np.abs(o64["m"][p]) + 1.0))
            assert np.all(err[ok] <= bound[ok]), f"rule {rule} x vs fp64 tensor {p}"
        if broadcast:
            # Every replica equals x on the tensors' elements (padding untouched).
            for i in range(n):
                for a, b in zip(ar.views(ar.replica(i)), ar.views(ar.x)):
                    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    ar.destroy()
    return nonbit


@pytest.mark.parametrize("rule", [dsm.DSM_RULE_LOOKAHEAD, dsm.DSM_RULE_SIGNED_SLOWMO,
                                  dsm.DSM_RULE_GLOBAL_ADAMW])
@pytest.mark.parametrize("n,broadcast", [(1, True), (3, True), (4, False), (5, True)])
@pytest.mark.parametrize("layout", [dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED,
                                    dsm.DSM_REPLICAS_STATE_BLOCKED])
def test_global_variant_parity(rule, n, broadcast, layout):
    nonbit = _run_variant(rule, n, broadcast, rounds=3, seed=31 * n + rule, layout=layout)
    print(f"rule {rule} n={n}: {nonbit} elements not bit-identical to the fp32 oracle")
    assert nonbit == 0


def test_variant_argument_errors():
    ar = A.Arenas([100, 7], 2, 1, dsm.DSM_BASE_SGD_MOMENTUM, randomized=True)
    ar.init()
    dsm.dsm_local_step(ar.ctx, -1, 1, **SGD)
    for kw, status in ((dict(rule=dsm.DSM_RULE_LOOKAHEAD, mode=dsm.DSM_SIGN_RAND_FLIP),
                        dsm.DSM_ERR_INVALID_ARG),
                       (dict(rule=dsm.DSM_RULE_GLOBAL_ADAMW), dsm.DSM_ERR_INVALID_ARG),  # no v
                       (dict(rule=7), dsm.DSM_ERR_INVALID_ARG)):
        with pytest.raises(dsm.DsmError) as e:
            dsm.dsm_global_step(ar.ctx, 0, **GLOB, **kw)
        assert e.value.status == status
    dsm.dsm_sync(ar.ctx)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_round_end(ar.ctx, 1, SGD, 0, rule=dsm.DSM_RULE_LOOKAHEAD, **GLOB)
    assert e.value.status == dsm.DSM_ERR_UNSUPPORTED
    dsm.dsm_round_end(ar.ctx, 1, SGD, 0, **GLOB)
    ar.destroy()
