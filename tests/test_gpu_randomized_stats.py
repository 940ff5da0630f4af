"""Lemma 1 on the GPU path at scale: the randomized sign is unbiased.

Section 3.1, Lemma 1: for either randomized sign, E[S_r(u)] = u/B.  The
variance is 1 - (u/B)^2 for Eq. (9) and |u|/B - (u/B)^2 for Eq. (10).

The inputs make u exact and S directly readable:
  * x = 0 and one worker;
  * one SGD local step with lr = 1 and no momentum, so x_1 = -g;
  * a global step with beta1 = 0 and gamma = eta = 1, so u = g and
    x_new = -S.
The gradient plants 2^21 elements in each of eight classes u/B in
{1, 0.75, 0.5, 0.25, 0.1, 0, -0.5, -1}.  Per class, the mean of S must lie
within 5 standard errors of u/B, and the sample variance near its expected
value.  The limits are exact: |u| = B always keeps sign(u), and u = 0 gives
S = 0.  The split global step and the fused round end (H = 1) both draw.
"""
import numpy as np
import pytest
import torch

from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

CLASSES = np.array([1.0, 0.75, 0.5, 0.25, 0.1, 0.0, -0.5, -1.0], dtype=np.float32)
N = 1 << 24


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
@pytest.mark.parametrize("mode", [dsm.DSM_SIGN_RAND_FLIP, dsm.DSM_SIGN_RAND_ZERO])
@pytest.mark.parametrize("seed", [1, 0xDEADBEEFCAFE])
def test_randomized_sign_is_unbiased_at_scale(mode, seed, fused):
    ar = A.Arenas([N], 1, 1, dsm.DSM_BASE_SGD_MOMENTUM, decay=[False], randomized=True)
    ar.x.zero_()
    ar.init()
    cls = torch.arange(N, device="cuda") % len(CLASSES)
    g = torch.as_tensor(CLASSES, device="cuda")[cls]
    ar.g_rep[0, :N] = g
    glob = dict(gamma=1.0, eta=1.0, beta1=0.0, beta2=0.5, lam=0.0, mode=mode, seed=seed,
                broadcast=True)
    if fused:
        dsm.dsm_round_end(ar.ctx, 1, dict(lr=1.0, beta1=0.0), 5, **glob)
    else:
        dsm.dsm_local_step(ar.ctx, -1, 1, lr=1.0, beta1=0.0)
        dsm.dsm_global_step(ar.ctx, 5, **glob)
    torch.cuda.synchronize()
    u = ar.u[:N].cpu().numpy()
    S = -ar.x[:N].cpu().numpy()
    B = dsm.dsm_read_bounds(ar.ctx, 1)[0]
    assert B == 1.0
    np.testing.assert_array_equal(u, g.cpu().numpy())       # u = g exactly
    assert set(np.unique(S)).issubset({-1.0, 0.0, 1.0})
    c = cls.cpu().numpy()
    for k, r in enumerate(CLASSES.astype(np.float64)):
        s = S[c == k].astype(np.float64)
        if abs(r) == 1.0:
            assert np.all(s == np.sign(r)), f"|u| = B must keep sign(u) (class {r})"
            continue
        if r == 0.0:
            assert np.all(s == 0.0), "u = 0 must give S = 0"
            continue
        var = 1.0 - r * r if mode == dsm.DSM_SIGN_RAND_FLIP else abs(r) - r * r
        se = np.sqrt(var / s.size)
        assert abs(s.mean() - r) < 5 * se, (mode, r, s.mean(), se)
        assert abs(s.var() - var) < 0.01, (mode, r, s.var(), var)
        if mode == dsm.DSM_SIGN_RAND_FLIP:
            assert not np.any(s == 0.0)                   # Eq. (9) never gives 0 off zero
        else:
            assert not np.any(s == -np.sign(r))           # Eq. (10) never flips
    ar.destroy()
