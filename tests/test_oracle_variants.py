"""Pins of the oracle's global-step variants (Section 4.1, Appendix C).

Lookahead reduces to the slow-weight interpolation of the Lookahead
optimizer; signed SlowMo with beta1 = 0 is a sign step on the averaged
difference; Global AdamW (Algorithm 7) is AdamW on the pseudo-gradient,
checked against torch.optim.AdamW and against its constant-gradient closed
form.
"""
import numpy as np
import pytest
import torch

import oracle as O


def _setup(rng, n, d=777, spread=1e-3):
    x = rng.normal(0, 0.02, d).astype(np.float32)
    m = rng.normal(0, 1, d).astype(np.float32)
    reps = [(x + rng.normal(0, spread, d)).astype(np.float32) for _ in range(n)]
    return x, m, reps


@pytest.mark.parametrize("n", [1, 3])
def test_lookahead_is_slow_weight_interpolation(n):
    """beta1 = beta2 = 0, lambda = 0: x' = x + eta (mean_i x_i - x), the
    Lookahead optimizer's slow-weight update with step eta."""
    rng = np.random.default_rng(1)
    x, m, reps = _setup(rng, n)
    res = O.global_step([x], [m], [[r] for r in reps], gamma=0.125, eta=0.5, beta1=0.0,
                        beta2=0.0, lam=0.0, decay=[True], rule=O.RULE_LOOKAHEAD)
    avg = np.mean(np.stack(reps).astype(np.float64), axis=0)
    expect = x + 0.5 * (avg - x)
    np.testing.assert_allclose(res["x"][0], expect, rtol=1e-14, atol=1e-17)
    assert res["S"][0] is None


@pytest.mark.parametrize("prec", ["fp64", "fp32"])
def test_lookahead_steps_along_the_momentum(prec):
    """beta1 = beta2: u = m_{t+1} and x' = x - eta gamma (m_{t+1} + lambda x)."""
    rng = np.random.default_rng(2)
    x, m, reps = _setup(rng, 4)
    kw = dict(gamma=1e-3, eta=0.8, beta1=0.9, beta2=0.9, lam=0.1, decay=[True], prec=prec)
    res = O.global_step([x], [m], [[r] for r in reps], rule=O.RULE_LOOKAHEAD, **kw)
    np.testing.assert_array_equal(res["u"][0], res["m"][0])
    ref = O.global_step([x], [m], [[r] for r in reps], **kw)
    np.testing.assert_array_equal(res["m"][0], ref["m"][0])
    dt = O.PRECISIONS[prec]
    s = dt(O.f32(0.8) * O.f32(1e-3))
    np.testing.assert_array_equal(res["x"][0], x.astype(dt) - s * (res["m"][0] + dt(O.f32(0.1)) * x.astype(dt)))


@pytest.mark.parametrize("prec", ["fp64", "fp32"])
def test_signed_slowmo_without_momentum_is_a_sign_step(prec):
    """beta1 = 0, lambda = 0, gamma dyadic: x' = x - eta sign(x - mean_i x_i)
    exactly; the momentum is Eq. (8) of the unsigned difference."""
    rng = np.random.default_rng(3)
    x, m, reps = _setup(rng, 2)
    reps[0][:50] = x[:50]
    reps[1][:50] = x[:50]            # zero difference -> sign 0 -> no move
    kw = dict(gamma=0.125, eta=0.25, beta1=0.0, beta2=0.9, lam=0.0, decay=[True], prec=prec)
    res = O.global_step([x], [m], [[r] for r in reps], rule=O.RULE_SIGNED_SLOWMO, **kw)
    avg = np.mean(np.stack(reps).astype(np.float64), axis=0)
    expect = x - 0.25 * np.sign(x - avg)
    np.testing.assert_array_equal(res["x"][0], expect.astype(O.PRECISIONS[prec]))
    np.testing.assert_array_equal(res["x"][0][:50], x[:50])
    ref = O.global_step([x], [m], [[r] for r in reps], **kw)
    np.testing.assert_array_equal(res["m"][0], ref["m"][0])


def test_signed_slowmo_combines_old_momentum_and_signed_difference():
    """u = beta1 m + (1 - beta1)/gamma sign(delta), with dyadic numbers exact."""
    x = np.array([1.0, -1.0, 0.5, 0.25], dtype=np.float32)
    m = np.array([2.0, 2.0, -4.0, 0.0], dtype=np.float32)
    reps = [np.array([0.5, -0.5, 0.5, 0.0], dtype=np.float32)]
    res = O.global_step([x], [m], [reps], gamma=0.25, eta=0.5, beta1=0.5, beta2=0.5, lam=0.0,
                        decay=[False], rule=O.RULE_SIGNED_SLOWMO)
    # delta = [0.5, -0.5, 0, 0.25]; sign = [1, -1, 0, 1]; (1-b1)/gamma = 2
    np.testing.assert_array_equal(res["u"][0], [3.0, -1.0, -2.0, 2.0])
    np.testing.assert_array_equal(res["x"][0], x - 0.125 * np.array([3.0, -1.0, -2.0, 2.0]))
    np.testing.assert_array_equal(res["m"][0], [2.0, 0.0, -2.0, 0.5])


def test_global_adamw_matches_torch_adamw_on_the_pseudo_gradient():
    """Algorithm 7 over several rounds: AdamW with lr eta on g_t =
    (x_{t,0} - x_{t,tau})/gamma_t, bias corrections 1 - beta^(t+1)."""
    rng = np.random.default_rng(4)
    d, n = 2049, 3
    b1, b2, eps, eta, lam, gamma = (O.f32(v) for v in (0.9, 0.95, 1e-8, 1e-3, 0.1, 2e-4))
    x = rng.normal(0, 0.02, d).astype(np.float32)
    m = np.zeros(d, np.float32)
    v = np.zeros(d, np.float32)
    for t in range(4):
        reps = [(x - rng.normal(0, 1e-4, d)).astype(np.float32) for _ in range(n)]
        res = O.global_step([x], [m], [[r] for r in reps], gamma=gamma, eta=eta, beta1=b1,
                            beta2=b2, lam=lam, eps=eps, decay=[True], t=t,
                            rule=O.RULE_GLOBAL_ADAMW, v=[v])
        # Pseudo-gradient of Algorithm 7 (the differences x - x_i are exact in
        # fp64, so their mean carries one rounding).
        g = np.mean(x.astype(np.float64) - np.stack(reps).astype(np.float64), axis=0) / gamma
        p = torch.nn.Parameter(torch.tensor(x, dtype=torch.float64))
        opt = torch.optim.AdamW([p], lr=eta, betas=(b1, b2), eps=eps, weight_decay=lam,
                                foreach=False)
        opt.state[p] = {"step": torch.tensor(float(t)),
                        "exp_avg": torch.tensor(m, dtype=torch.float64),
                        "exp_avg_sq": torch.tensor(v, dtype=torch.float64)}
        p.grad = torch.tensor(g)
        opt.step()
        np.testing.assert_allclose(res["m"][0], opt.state[p]["exp_avg"].numpy(), rtol=1e-12,
                                   atol=1e-12)
        np.testing.assert_allclose(res["v"][0], opt.state[p]["exp_avg_sq"].numpy(), rtol=1e-12)
        np.testing.assert_allclose(res["x"][0], p.detach().numpy(), rtol=1e-13, atol=1e-16)
        x, m, v = (a.astype(np.float32) for a in (res["x"][0], res["m"][0], res["v"][0]))


@pytest.mark.parametrize("decayed", [True, False])
def test_global_adamw_constant_pseudo_gradient_closed_form(decayed):
    """Constant g: m_hat = g and v_hat = g^2, so x' = x - eta (g/(|g|+eps) + lambda x),
    with lambda = 0 on a tensor whose decay flag is off."""
    rng = np.random.default_rng(5)
    d = 500
    x0 = rng.normal(0, 0.02, d).astype(np.float32)
    # Differences bounded away from 0, so the fp32 rounding of the replicas
    # barely moves g between rounds.
    diff = (np.sign(rng.normal(size=d)) * (1e-3 + np.abs(rng.normal(0, 1e-3, d)))).astype(np.float32)
    gamma, eta, lam, eps = 0.125, 1e-2, 0.1, 1e-8
    st = O.init_state([x0], 1, "sgd")
    x, m, v = x0, np.zeros(d, np.float32), np.zeros(d, np.float32)
    for t in range(5):
        rep = (x - diff).astype(np.float32)
        res = O.global_step([x], [m], [[rep]], gamma=gamma, eta=eta, beta1=0.9, beta2=0.95,
                            lam=lam, eps=eps, decay=[decayed], t=t, rule=O.RULE_GLOBAL_ADAMW,
                            v=[v])
        g = (x.astype(np.float64) - rep) / gamma
        lam_p = O.f32(lam) if decayed else 0.0
        expect = x - O.f32(eta) * (g / (np.abs(g) + O.f32(eps)) + lam_p * x)
        # The replicas are rounded to fp32, so g varies by ~1e-6 relative between
        # rounds; a wrong bias correction would move x by O(eta).
        np.testing.assert_allclose(res["x"][0], expect, rtol=1e-9, atol=1e-5 * eta)
        x, m, v = (a.astype(np.float32) for a in (res["x"][0], res["m"][0], res["v"][0]))
    del st


def test_variants_reject_the_randomized_sign():
    x, m, reps = _setup(np.random.default_rng(6), 2, d=10)
    for rule in (O.RULE_LOOKAHEAD, O.RULE_SIGNED_SLOWMO, O.RULE_GLOBAL_ADAMW):
        with pytest.raises(ValueError):
            O.global_step([x], [m], [[r] for r in reps], gamma=1e-3, eta=1.0, beta1=0.9,
                          beta2=0.9, lam=0.0, decay=[True], mode=O.SIGN_RAND_FLIP, rule=rule,
                          v=[np.zeros_like(x)])


def test_global_adamw_round_driver_keeps_v():
    """communication_round carries the Global AdamW second moment across rounds."""
    rng = np.random.default_rng(7)
    x0 = [rng.normal(0, 0.02, 64).astype(np.float32)]
    st = O.init_state(x0, 2, "sgd")
    g = [[rng.normal(0, 1e-2, 64).astype(np.float32)] for _ in range(2)]
    glob = dict(eta=1e-3, beta1=0.9, beta2=0.95, lam=0.0, eps=1e-8, mode=O.SIGN_DET, seed=0,
                rule=O.RULE_GLOBAL_ADAMW)
    for t in range(3):
        O.communication_round(st, lambda i, k: g[i], t, H=2, local=dict(lr=0.01, beta1=0.0),
                              glob=glob, decay=[True])
    assert "v" in st and np.all(st["v"][0] > 0)


def test_global_adamw_round_driver_closed_form():
    """Through the round driver (Algorithm 1, SGD base without momentum, the
    same gradient g on every worker at every local step): the pseudo-gradient
    of every round is the constant (x - x_i)/gamma = H g, so Algorithm 7 moves
    x by eta (Hg/(|Hg|+eps) + lambda x) in every round, which holds only if
    round t gets the bias corrections 1 - beta^(t+1)."""
    rng = np.random.default_rng(11)
    d = 256
    x0 = rng.normal(0, 0.02, d).astype(np.float32)
    g = (np.sign(rng.normal(size=d)) * (1e-2 + np.abs(rng.normal(0, 1e-2, d)))).astype(np.float32)
    H, lr, eta, lam, eps = 2, 0.125, 1e-3, 0.1, 1e-8
    st = O.init_state([x0], 2, "sgd")
    glob = dict(eta=eta, beta1=0.9, beta2=0.95, lam=lam, eps=eps, mode=O.SIGN_DET, seed=0,
                rule=O.RULE_GLOBAL_ADAMW)
    for t in range(4):
        x = st["x"][0].astype(np.float64)
        O.communication_round(st, lambda i, k: [g], t, H=H, local=dict(lr=lr, beta1=0.0),
                              glob=glob, decay=[True])
        G = H * g.astype(np.float64)
        expect = x - O.f32(eta) * (G / (np.abs(G) + O.f32(eps)) + O.f32(lam) * x)
        # fp32 replicas move G by ~1e-6 relative; a bias correction of the
        # wrong round moves the step by 10% or more.
        np.testing.assert_allclose(st["x"][0], expect, rtol=0, atol=1e-4 * eta)
