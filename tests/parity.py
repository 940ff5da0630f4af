"""Comparison helpers for the GPU parity tests (GPU path vs CPU oracle).

Two bars, per output element:
  * Against the oracle evaluated in fp32 (the GPU path's arithmetic type):
    |gpu - ora32| <= 1e-6 |ora32|, the stated 1e-6 relative tolerance; the
    number of elements that are not bit-identical is reported (expected 0).
    Integer outputs (signs, Philox words, replica copies) are compared
    bit-exactly.
  * Against the oracle evaluated in fp64: |gpu - ora64| <= K u S, where
    u = 2^-24, S is the element's magnitude scale (the same formula evaluated
    on absolute values: a running error bound), and K = 32 is twice the
    number of fp32 roundings on the longest operation chain (16, AdamW).
    Sign decisions may differ from fp64 only where the fp64 decision margin is
    below 1e-6 * rms of u over the tensor; those flips are counted and the
    flipped elements' x is excluded.  For the randomized sign the margin is
    the distance of |u| from the Eq. (9) / Eq. (10) threshold, both sides
    drawing the same Philox words.
"""
import numpy as np

U32 = 2.0 ** -24
K_ROUNDINGS = 32
RTOL = 1e-6


def rel_check(gpu, ora, what, rtol=RTOL):
    """Strict relative check; returns the count of non-bit-identical elements."""
    g = np.asarray(gpu, dtype=np.float64)
    o = np.asarray(ora, dtype=np.float64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    both_nan = np.isnan(g) & np.isnan(o)
    err = np.abs(g - o)
    bad = ~both_nan & ~(err <= rtol * np.abs(o))
    if bad.any():
        i = np.flatnonzero(bad)[:5]
        raise AssertionError(f"{what}: {bad.sum()} of {g.size} elements differ by more than "
                             f"{rtol} relative; first at {i}: gpu {g[i]} oracle {o[i]}")
    gb = np.asarray(gpu, dtype=np.float32).view(np.uint32)
    ob = np.asarray(ora, dtype=np.float32).view(np.uint32)
    return int(np.count_nonzero(gb != ob))


def scaled_check(gpu, ora64, scale, what, mask=None):
    """|gpu - ora64| <= K u scale on the elements of mask (default all)."""
    g = np.asarray(gpu, dtype=np.float64)
    o = np.asarray(ora64, dtype=np.float64)
    tol = K_ROUNDINGS * U32 * np.asarray(scale, dtype=np.float64)
    bad = ~(np.abs(g - o) <= tol)
    if mask is not None:
        bad &= mask
    if bad.any():
        i = np.flatnonzero(bad)[:5]
        raise AssertionError(f"{what}: {bad.sum()} of {g.size} elements outside the fp64 "
                             f"error bound; first at {i}: gpu {g[i]} oracle64 {o[i]} "
                             f"bound {tol[i]}")


def adamw_scales(x, g, m, v, *, lr, beta1, beta2, eps, weight_decay, step, o64):
    """Magnitude scales of the AdamW outputs (m, v, x) for scaled_check."""
    import oracle as O
    x, g, m, v = (np.asarray(a, np.float64) for a in (x, g, m, v))
    b1, b2 = O.f32(beta1), O.f32(beta2)
    bc1 = 1.0 - O.beta_power(b1, step)
    bc2 = 1.0 - O.beta_power(b2, step)
    s_m = b1 * np.abs(m) + (1 - b1) * np.abs(g)
    s_v = np.asarray(o64[2], np.float64)
    den = np.sqrt(s_v / bc2) + O.f32(eps)
    s_x = np.abs(x) + O.f32(lr) * ((s_m / bc1) / den + O.f32(weight_decay) * np.abs(x))
    return s_m, s_v, s_x


def sgdm_scales(x, g, m, *, lr, momentum):
    import oracle as O
    x, g, m = (np.asarray(a, np.float64) for a in (x, g, m))
    s_m = O.f32(momentum) * np.abs(m) + np.abs(g)
    s_x = np.abs(x) + O.f32(lr) * s_m
    return s_m, s_x


def global_scales(x, m, reps, S, *, gamma, eta, beta1, beta2, lam_p):
    import oracle as O
    x = np.asarray(x, np.float64)
    m = np.asarray(m, np.float64)
    n = len(reps)
    s_d = sum(np.abs(x - np.asarray(r, np.float64)) for r in reps) / n
    g_ = O.f32(gamma)
    c1 = (1 - O.f32(beta1)) / g_
    c2 = (1 - O.f32(beta2)) / g_
    s_u = O.f32(beta1) * np.abs(m) + c1 * s_d
    s_m = O.f32(beta2) * np.abs(m) + c2 * s_d
    s_x = np.abs(x) + O.f32(eta) * g_ * (np.abs(S) + O.f32(lam_p) * np.abs(x))
    return s_u, s_m, s_x


FLIP_MARGIN = 1e-6


def det_flip_check(S32, S64, u64, rms_u, what):
    """Deterministic sign decisions of the fp32 oracle (bit-identical to the
    GPU path's, whose x is checked bit for bit) against the fp64 oracle's.
    A flip is allowed only where |u| < 1e-6 rms_p(u).  Returns the count."""
    s32, s64 = np.asarray(S32, np.float64), np.asarray(S64, np.float64)
    flip = ~((s32 == s64) | (np.isnan(s32) & np.isnan(s64)))
    if flip.any():
        au = np.abs(np.asarray(u64, np.float64)[flip])
        bad = ~(au < FLIP_MARGIN * rms_u)
        if bad.any():
            raise AssertionError(f"{what}: {bad.sum()} of {flip.sum()} sign flips vs fp64 lie "
                                 f"outside |u| < {FLIP_MARGIN} rms(u) = {FLIP_MARGIN * rms_u}: "
                                 f"|u| {au[bad][:5]}")
    return int(flip.sum())


def rand_flip_check(S32, S64, u64, B64, k, variant, rms_u, what):
    """Randomized sign decisions (Eq. (9) variant 1, Eq. (10) variant 2) of the
    fp32 oracle against the fp64 oracle's, both drawn with the same Philox
    words k (U = k 2^-24).  A decision may differ only where the fp64 decision
    margin is below 1e-6 rms_p(u): |u| (the sign of u itself), or the distance
    of |u| from the threshold, ||u| - B (2U - 1)| for Eq. (9) and ||u| - B U|
    for Eq. (10).  Returns the number of differing decisions."""
    s32, s64 = np.asarray(S32, np.float64), np.asarray(S64, np.float64)
    flip = ~((s32 == s64) | (np.isnan(s32) & np.isnan(s64)))
    if flip.any():
        au = np.abs(np.asarray(u64, np.float64)[flip])
        U = np.asarray(k, np.float64)[flip] * U32
        thr = float(B64) * ((2.0 * U - 1.0) if variant == 1 else U)
        margin = np.minimum(au, np.abs(au - thr))
        bad = ~(margin < FLIP_MARGIN * rms_u)
        if bad.any():
            raise AssertionError(f"{what}: {bad.sum()} of {flip.sum()} randomized decisions "
                                 f"differ from fp64 with margin >= {FLIP_MARGIN} rms(u) = "
                                 f"{FLIP_MARGIN * rms_u}: margins {margin[bad][:5]}")
    return int(flip.sum())


def rms(a):
    a = np.asarray(a, np.float64)
    return float(np.sqrt(np.mean(a * a))) if a.size else 0.0
