"""Checkpoint and resume at a round boundary are bitwise exact.

All of the method's state lives in caller-owned buffers: x, m, the base
optimizer's per-worker state, and v for Global AdamW.  The counters are
explicit arguments: s and t.  The randomized sign draws from Philox keyed by
(seed, t, tensor, element).  So a run can be resumed at a round boundary in a
fresh allocation:
  1. write the saved x;
  2. call dsm_init, which sets the replicas to x and zeroes the rest;
  3. write back m, s1, s2 and v;
  4. continue with the saved counters.
The replicas need no saving: after a global step they equal x, or they are
stale after a lazy broadcast, which is the same thing.
"""
import numpy as np
import pytest
import torch

from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

NUMEL = [1, 5, 64, 65, 1000, 16385, 40003]
DECAY = [i % 2 == 0 for i in range(len(NUMEL))]
N, H = 3, 3
LOCAL = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
GLOB = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1, seed=0xABCDEF0123)
# Round t: (sign mode, fused round end with lazy broadcast or split with broadcast).
ROUNDS = [(dsm.DSM_SIGN_RAND_FLIP, True), (dsm.DSM_SIGN_DET, False),
          (dsm.DSM_SIGN_RAND_ZERO, True), (dsm.DSM_SIGN_DET, True), (dsm.DSM_SIGN_RAND_FLIP, False)]
CUT = 2  # checkpoint after rounds 0 .. CUT-1


def grads(ar, t, k):
    gen = torch.Generator(device="cuda").manual_seed(7919 * t + 31 * k + 1)
    ar.g_rep.normal_(0.0, 1e-3, generator=gen)


def run_round(ar, t):
    mode, fused = ROUNDS[t]
    for k in range(H):
        grads(ar, t, k)
        s = t * H + k + 1
        if fused and k == H - 1:
            dsm.dsm_round_end(ar.ctx, s, LOCAL, t, mode=mode, broadcast=False, **GLOB)
        else:
            dsm.dsm_local_step(ar.ctx, -1, s, **LOCAL)
    if not fused:
        dsm.dsm_global_step(ar.ctx, t, mode=mode, broadcast=True, **GLOB)


# All three replica layouts: the ABI default, blocked replicas, and the
# bench's (replicas and their state blocked).
LAYOUTS = [dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED, dsm.DSM_REPLICAS_STATE_BLOCKED]


def fresh(seed, layout):
    ar = A.Arenas(NUMEL, N, H, dsm.DSM_BASE_ADAMW, decay=DECAY, randomized=True,
                  replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    ar.x.normal_(0.0, 0.02, generator=gen)
    return ar


def bits(ar, t):
    torch.cuda.synchronize()
    return np.concatenate([v.detach().cpu().numpy().view(np.uint32).ravel()
                           for v in ar.views(t)])


def final_state(ar):
    dsm.dsm_sync(ar.ctx)
    out = {"x": bits(ar, ar.x), "m": bits(ar, ar.m)}
    for name in ("x_rep", "s1_rep", "s2_rep"):
        for i in range(N):
            out[f"{name}[{i}]"] = bits(ar, ar.worker(name, i))
    return out


@pytest.mark.parametrize("layout", LAYOUTS)
def test_resume_at_round_boundary_is_bitwise_exact(layout):
    # Uninterrupted run, with the checkpoint taken on the way.
    ar = fresh(11, layout)
    ar.init()
    ckpt = None
    for t in range(len(ROUNDS)):
        if t == CUT:
            torch.cuda.synchronize()
            ckpt = {name: getattr(ar, name).detach().clone().cpu()
                    for name in ("x", "m", "s1_rep", "s2_rep")}
        run_round(ar, t)
    want = final_state(ar)
    ar.destroy()
    del ar
    # Resume in a fresh allocation (different addresses and placement).
    filler = torch.empty(12345, device="cuda")  # shifts the allocator
    ar = fresh(999, layout)
    ar.x.copy_(ckpt["x"].to("cuda"))
    ar.init()
    for name in ("m", "s1_rep", "s2_rep"):
        getattr(ar, name).copy_(ckpt[name].to("cuda"))
    for t in range(CUT, len(ROUNDS)):
        run_round(ar, t)
    got = final_state(ar)
    ar.destroy()
    del filler
    for key in want:
        assert np.array_equal(got[key], want[key]), f"{key} differs after resume"


@pytest.mark.parametrize("layout", LAYOUTS)
def test_resume_after_lazy_round_end(layout):
    """The cut falls right after a fused round end without broadcast, where
    the replicas on the device still hold the previous round's values."""
    cut = 1  # round 0 is fused and lazy
    assert ROUNDS[cut - 1][1]
    ar = fresh(3, layout)
    ar.init()
    run_round(ar, 0)
    torch.cuda.synchronize()
    ckpt = {name: getattr(ar, name).detach().clone() for name in ("x", "m", "s1_rep", "s2_rep")}
    stale = any(not torch.equal(a, b) for a, b in zip(ar.views(ar.replica(0)), ar.views(ar.x)))
    assert stale, "the lazy round end left the replicas as they were"
    for t in range(cut, 3):
        run_round(ar, t)
    want = final_state(ar)
    ar.destroy()
    ar = fresh(4, layout)
    ar.x.copy_(ckpt["x"])
    ar.init()
    for name in ("m", "s1_rep", "s2_rep"):
        getattr(ar, name).copy_(ckpt[name])
    for t in range(cut, 3):
        run_round(ar, t)
    got = final_state(ar)
    ar.destroy()
    for key in want:
        assert np.array_equal(got[key], want[key]), f"{key} differs after resume"
