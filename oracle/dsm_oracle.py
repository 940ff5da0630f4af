"""Plain CPU oracle of distributed sign momentum with local steps.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or run this module.  It shares no
code with the HIP library (no kernels, headers, tables or helpers) and never
imports it.

What it computes (arXiv 2411.17866):
  * Section 2, Eq. (4) and Algorithm 1: every worker i takes tau local steps
    x_{t,k+1}^(i) = x_{t,k}^(i) - gamma_t d_{t,k}^(i) with a base optimizer:
    AdamW (Algorithm 2, Appendix A) or SGD with Polyak momentum
    (Algorithm 3, Appendix A).
  * Algorithm 1, all-reduce and global step: the replicas are averaged and
    the global sign-momentum step of Eqs. (6)-(8) is taken:
        u_{t+1}   = beta1 m_t + (1-beta1)/gamma_t (x_{t,0} - x_{t,tau})
        x_{t+1,0} = x_{t,0} - eta gamma_t (sign(u_{t+1}) + lambda x_{t,0})
        m_{t+1}   = beta2 m_t + (1-beta2)/gamma_t (x_{t,0} - x_{t,tau})
    then every replica is reset to x_{t+1,0} (synchronisation step).
  * Section 3.1, Eqs. (9) and (10): the randomized sign operators S_r that
    the analysis uses in place of sign (Lemma 1: E[S_r(v)] = v/B).

Precision.  The paper fixes no arithmetic precision; the workload stores
every state buffer in fp32.  Each function evaluates its update in the
precision ``prec`` names, one IEEE round-to-nearest operation per written
operation, in the order the formula is written:
  * "fp64" (default): the accuracy reference.
  * "fp32": the same formula evaluated in fp32, the arithmetic type of the
    GPU path.  Decisions that floating point takes (the sign of u) are
    compared against this mode, in the GPU path's precision.
Hyperparameters are fp32 numbers (the library's arguments are fp32).
Scalar coefficients that depend only on hyperparameters (1 - beta^s,
(1-beta)/gamma, eta*gamma) are formed in fp64 and rounded once to the
working precision.  Results are returned in the working precision; the
round driver stores state as fp32 between steps.

Readings where the paper is silent (each is listed in the design notes):
  * sign(0) = 0.  Fixed by the proof of Theorem 3 (Appendix B.3), which
    starts from x_{0,0} = x_{-1,0} - eta gamma sign(m_0) with m_0 = 0 and
    concludes x_{0,0} = x_{-1,0}.
  * x_{t,0} - x_{t,tau} is formed as (1/n) sum_i (x_{t,0} - x_{t,tau}^(i)),
    summed in worker order i = 0..n-1 and divided by n: equal in exact
    arithmetic to subtracting the all-reduce average, and free of the
    cancellation of averaging first.
  * u_{t+1} and m_{t+1} both use the old m_t (Eqs. (6) and (8)).
  * Base-optimizer state (AdamW m, v; Polyak m) stays per worker, is never
    averaged or reset, and the bias-correction step s counts across rounds.
  * Weight decay (local and global) applies only to tensors whose decay flag
    is set; the flag selects lambda or 0 for the tensor.
  * The randomized bound B is max_j |u_j| over the tensor (the tightest
    bound for which Eqs. (9)/(10) are probabilities); B = 0 gives S = 0.  A
    bound that is not finite leaves S_r undefined (Section 3.1 needs a finite
    B): S is NaN over the whole tensor.
  * Random uniforms: U = (w >> 8) * 2^-24 from Philox4x32-10 with key = seed
    and counter (j div 4, tensor index, t, 1), word j mod 4, where j is the
    element's index inside its tensor.  "w.p. p" is the exact comparison
    U < p.

Parity unpinned: every function here is checked against independent facts
(worked examples, closed forms, library and textbook reductions, Monte Carlo
of Lemma 1, a Philox known-answer test), but these aspects are fixed by the
readings above, not by the paper, and no pin can tie them to it: the worker
order of the difference form (pinned only up to rounding), the persistence
of the base-optimizer state and of s across rounds, the Philox stream
layout, and the momentum of the signed-SlowMo variant (Section 4.1).
"""
from fractions import Fraction

import numpy as np

from .philox import philox4x32_10

PRECISIONS = {"fp64": np.float64, "fp32": np.float32}

SIGN_DET = 0
SIGN_RAND_FLIP = 1   # Eq. (9): -sign w.p. 1/2 - |v|/2B, sign w.p. 1/2 + |v|/2B
SIGN_RAND_ZERO = 2   # Eq. (10): 0 w.p. 1 - |v|/B, sign w.p. |v|/B

PHILOX_STREAM = 1    # fourth counter word of the randomized-sign stream

# Global-step rules: the method's sign momentum and the ablation variants of
# Section 4.1 and Appendix C.
RULE_SIGN_MOMENTUM = 0   # Eqs. (6)-(8)
RULE_LOOKAHEAD = 1       # Eq. (7) replaced by x - eta gamma u (Section 4.1)
RULE_SIGNED_SLOWMO = 2   # Eqs. (6), (7) with sign on the difference (Section 4.1)
RULE_GLOBAL_ADAMW = 3    # Algorithm 7 (Appendix C)
_TWO24 = 16777216.0


def _dtype(prec):
    try:
        return PRECISIONS[prec]
    except KeyError:
        raise ValueError(f"prec must be one of {sorted(PRECISIONS)}") from None


def f32(h):
    """A hyperparameter as the fp32 number the library receives."""
    return float(np.float32(h))


def beta_power(beta, s):
    """beta**s in fp64 by binary exponentiation (square and multiply, lowest
    bit of s first): O(log s) operations for any s and any beta in [0, 1]."""
    result, base, e = 1.0, float(beta), int(s)
    while e > 0:
        if e & 1:
            result *= base
        base *= base
        e >>= 1
    return result


# --------------------------------------------------------------------------
# Local base-optimizer steps (Algorithm 1 inner loop, Eq. (4))
# --------------------------------------------------------------------------

def local_adamw_step(x, g, m, v, *, lr, beta1, beta2, eps, weight_decay, step,
                     prec="fp64"):
    """One AdamW step (Algorithm 2, Appendix A) on one tensor of one worker.

    x, g, m, v: arrays of one tensor (fp32 storage).  ``step`` is the
    bias-correction count s >= 1 (the t+1 of Algorithm 2).  ``weight_decay``
    is lambda for this tensor (0 when the tensor is not decayed).  The local
    learning rate gamma_t of Eq. (4) is ``lr``.  Returns (x, m, v).
    """
    dt = _dtype(prec)
    if step < 1:
        raise ValueError("bias-correction step must be >= 1")
    x, g, m, v = (np.asarray(a, dtype=np.float32).astype(dt) for a in (x, g, m, v))
    b1, b2 = f32(beta1), f32(beta2)
    beta1_, beta2_ = dt(b1), dt(b2)
    one_minus_b1 = dt(1.0 - b1)
    one_minus_b2 = dt(1.0 - b2)
    bc1 = dt(1.0 - beta_power(b1, step))
    bc2 = dt(1.0 - beta_power(b2, step))
    lr_, eps_, wd_ = dt(f32(lr)), dt(f32(eps)), dt(f32(weight_decay))

    # Momentum updates.
    m_new = beta1_ * m + one_minus_b1 * g
    v_new = beta2_ * v + one_minus_b2 * (g * g)
    # Bias corrections.
    m_hat = m_new / bc1
    v_hat = v_new / bc2
    # Parameter update with decoupled weight decay on the old x.
    x_new = x - lr_ * (m_hat / (np.sqrt(v_hat) + eps_) + wd_ * x)
    return x_new, m_new, v_new


def local_sgdm_step(x, g, m, *, lr, momentum, prec="fp64"):
    """One SGD step with Polyak momentum (Algorithm 3, Appendix A).

    m <- beta m + g;  x <- x - lr m   (no dampening, no Nesterov term).
    Returns (x, m).
    """
    dt = _dtype(prec)
    x, g, m = (np.asarray(a, dtype=np.float32).astype(dt) for a in (x, g, m))
    mu = dt(f32(momentum))
    lr_ = dt(f32(lr))
    m_new = mu * m + g
    x_new = x - lr_ * m_new
    return x_new, m_new


# --------------------------------------------------------------------------
# Global step (Algorithm 1: all-reduce, Eqs. (6)-(8), synchronisation)
# --------------------------------------------------------------------------

def sign(u):
    """sign with sign(+-0) = +0 (Appendix B.3) and sign(NaN) = NaN."""
    return np.sign(u) + u.dtype.type(0.0)


def randomized_sign_uniforms(numel, tensor_index, t, seed):
    """The integer k = w >> 8 (so U = k * 2^-24) for every element of a tensor.

    Philox4x32-10 keyed by the 64-bit seed (low word k0, high word k1) with
    counter (j div 4, tensor_index, t, 1); element j takes word j mod 4.
    """
    if not (0 <= t < 2 ** 32):
        raise ValueError("t must be in [0, 2^32)")
    if not (0 <= tensor_index < 2 ** 32):
        raise ValueError("tensor index must be in [0, 2^32)")
    nblk = (numel + 3) // 4
    q = np.arange(nblk, dtype=np.uint64)
    w = philox4x32_10(q, tensor_index, t, PHILOX_STREAM,
                      seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    words = np.stack(w, axis=1).reshape(-1)[:numel]
    return (words >> np.uint32(8)).astype(np.int64)


def randomized_sign_uniforms_at(j, tensor_index, t, seed):
    """k = w >> 8 for chosen element indices j of a tensor (same stream as
    randomized_sign_uniforms, evaluated only where asked)."""
    if not (0 <= t < 2 ** 32):
        raise ValueError("t must be in [0, 2^32)")
    j = np.asarray(j, dtype=np.uint64)
    w = philox4x32_10(j >> np.uint64(2), tensor_index, t, PHILOX_STREAM,
                      seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    words = np.stack(w, axis=1)
    pick = words[np.arange(j.size), (j & np.uint64(3)).astype(np.int64)]
    return (pick >> np.uint32(8)).astype(np.int64)


def _exact_less(a_int, B, au):
    """Elementwise exact test  a_int * B < au * 2^24  for integers a_int.

    a_int: int64 array with |a_int| <= 2^24; B: finite scalar >= 0; au: array
    >= 0.  Evaluated in fp64; every element whose two finite sides are within
    a relative 2^-45 of each other is re-decided with exact rationals.  Where
    u is infinite or NaN the fp64 comparison is already the IEEE one:
    infinities compare exactly and NaN compares false.
    """
    B = float(B)
    with np.errstate(invalid="ignore"):
        lhs = a_int.astype(np.float64) * B
        rhs = au.astype(np.float64) * _TWO24
        res = lhs < rhs
        close = (np.isfinite(lhs) & np.isfinite(rhs) &
                 (np.abs(lhs - rhs) <= 2.0 ** -45 * np.maximum(np.abs(lhs), np.abs(rhs))))
    if np.any(close):
        fb = Fraction(B)
        for idx in np.flatnonzero(close):
            res[idx] = Fraction(int(a_int[idx])) * fb < Fraction(float(au[idx])) * 16777216
    return res


def randomized_sign(u, B, k, variant):
    """S_r(u) of Eq. (9) (variant SIGN_RAND_FLIP) or Eq. (10) (SIGN_RAND_ZERO).

    u: array; B: the bound (scalar >= 0); k: integers with U = k 2^-24.
    Eq. (9): keep sign(u) w.p. 1/2 + |u|/(2B), i.e. iff U < 1/2 + |u|/(2B),
             i.e. (2k - 2^24) B < |u| 2^24; otherwise -sign(u).
    Eq. (10): keep sign(u) w.p. |u|/B, i.e. iff k B < |u| 2^24; otherwise 0.
    Both comparisons are exact.  u = 0 or B = 0 gives 0.

    Section 3.1 defines S_r only for a finite bound B >= |v_j|.  A bound that
    is NaN or infinite (B = max |u| over a tensor that holds a NaN or an
    infinite u_j) leaves the randomized sign of the whole tensor undefined:
    every element then gets NaN, so the tensor's step is NaN, as the
    deterministic sign makes it at a NaN u, and never a finite step of a
    reversed or zero sign.
    """
    dt = u.dtype.type
    if not np.isfinite(B):
        return np.full(np.shape(u), np.nan, dtype=u.dtype)
    s = sign(u)
    au = np.abs(u)
    if variant == SIGN_RAND_FLIP:
        keep = _exact_less(2 * k - (1 << 24), B, au)
        return np.where(keep, s, dt(0.0) - s)
    if variant == SIGN_RAND_ZERO:
        keep = _exact_less(k, B, au)
        return np.where(keep, s, dt(0.0))
    raise ValueError("unknown randomized-sign variant")


def global_step(x, m, replicas, *, gamma, eta, beta1, beta2, lam, decay,
                t=0, mode=SIGN_DET, seed=0, prec="fp64", tensor_ids=None,
                element_ids=None, bounds=None, rule=RULE_SIGN_MOMENTUM, v=None, eps=1e-8):
    """Algorithm 1 global step for a model given as a list of tensors.

    x:        list of arrays, x_{t,0} per tensor.
    m:        list of arrays, m_t per tensor.
    replicas: list over the n workers of lists of arrays, x_{t,tau}^(i).
    decay:    list of bools, whether lambda applies to each tensor.
    mode:     SIGN_DET, SIGN_RAND_FLIP (Eq. (9)) or SIGN_RAND_ZERO (Eq. (10)).
    t, seed:  outer iteration and 64-bit seed keying the randomized sign.
    Evaluating samples of tensors (every update is elementwise given B_p):
    tensor_ids:  tensor index p of each entry (default: its list position);
    element_ids: per entry, the in-tensor indices j of its elements (default:
                 the entry is the whole tensor, j = 0..numel-1);
    bounds:      per entry, B_p of the whole tensor (default: max |u| over
                 the entry, which is B_p when the entry is the whole tensor).

    rule:     the global update (deterministic sign only for the variants):
      RULE_SIGN_MOMENTUM  Eqs. (6)-(8).
      RULE_LOOKAHEAD      Section 4.1: Eq. (7) replaced by
                          x_{t+1,0} = x_{t,0} - eta gamma_t (u_{t+1} + lambda x_{t,0});
                          lambda = 0 is the paper's Lookahead.
      RULE_SIGNED_SLOWMO  Section 4.1: u_{t+1} = beta1 m_t + (1-beta1)/gamma_t
                          sign(x_{t,0} - x_{t,tau}); x_{t+1,0} = x_{t,0} - eta gamma_t
                          (u_{t+1} + lambda x_{t,0}); Eq. (8) unchanged.
      RULE_GLOBAL_ADAMW   Algorithm 7: AdamW on the pseudo-gradient
                          g_t = (1/gamma_t)(x_{t,0} - x_{t,tau}) with bias
                          corrections 1 - beta^(t+1), learning rate eta (not
                          scaled by gamma), epsilon eps and second moment v.

    Returns a dict of per-tensor lists: x (x_{t+1,0}), m (m_{t+1}), u
    (u_{t+1}; for Global AdamW the pseudo-gradient g_t), S (the sign actually
    applied; None for Lookahead and Global AdamW), delta ((x_{t,0}-x_{t,tau})),
    B (per-tensor bound, randomized modes only, else None) and v (Global AdamW
    only).
    """
    dt = _dtype(prec)
    n = len(replicas)
    if n < 1:
        raise ValueError("need at least one worker")
    b1, b2, g_ = f32(beta1), f32(beta2), f32(gamma)
    beta1_, beta2_ = dt(b1), dt(b2)
    c1 = dt((1.0 - b1) / g_)           # (1 - beta1) / gamma_t
    c2 = dt((1.0 - b2) / g_)           # (1 - beta2) / gamma_t
    step = dt(f32(eta) * g_)           # eta * gamma_t
    lam_ = dt(f32(lam))
    if rule != RULE_SIGN_MOMENTUM and mode != SIGN_DET:
        raise ValueError("the randomized sign applies to the sign-momentum rule only")
    if rule == RULE_GLOBAL_ADAMW:
        return _global_adamw(x, m, v, replicas, gamma=gamma, eta=eta, beta1=beta1, beta2=beta2,
                             lam=lam, eps=eps, decay=decay, t=t, dt=dt)
    out = {"x": [], "m": [], "u": [], "S": [], "delta": [], "B": None}
    if mode != SIGN_DET:
        out["B"] = []
    for p in range(len(x)):
        xp = np.asarray(x[p], dtype=np.float32).astype(dt)
        mp = np.asarray(m[p], dtype=np.float32).astype(dt)
        # All-reduce: (x_{t,0} - x_{t,tau}) = (1/n) sum_i (x_{t,0} - x^(i)).
        acc = xp - np.asarray(replicas[0][p], dtype=np.float32).astype(dt)
        for i in range(1, n):
            acc = acc + (xp - np.asarray(replicas[i][p], dtype=np.float32).astype(dt))
        delta = acc / dt(n)
        # Eq. (6) and Eq. (8), both from the old m_t.
        if rule == RULE_SIGNED_SLOWMO:
            u = beta1_ * mp + c1 * sign(delta)
        else:
            u = beta1_ * mp + c1 * delta
        m_new = beta2_ * mp + c2 * delta
        if rule in (RULE_LOOKAHEAD, RULE_SIGNED_SLOWMO):
            # The variants step along u itself (no sign).
            lam_p = lam_ if decay[p] else dt(0.0)
            out["x"].append(xp - step * (u + lam_p * xp))
            out["m"].append(m_new)
            out["u"].append(u)
            out["S"].append(None)
            out["delta"].append(delta)
            continue
        if mode == SIGN_DET:
            S = sign(u)
        else:
            pid = p if tensor_ids is None else int(tensor_ids[p])
            if bounds is not None:
                B = dt(bounds[p])
            else:
                B = np.max(np.abs(u)) if u.size else dt(0.0)
            if element_ids is None:
                k = randomized_sign_uniforms(u.size, pid, t, seed)
            else:
                k = randomized_sign_uniforms_at(element_ids[p], pid, t, seed)
            S = randomized_sign(u, B, k, mode)
            out["B"].append(dt(B))
        lam_p = lam_ if decay[p] else dt(0.0)
        # Eq. (7): decoupled weight decay on the old x_{t,0}.
        x_new = xp - step * (S + lam_p * xp)
        out["x"].append(x_new)
        out["m"].append(m_new)
        out["u"].append(u)
        out["S"].append(S)
        out["delta"].append(delta)
    return out


def _worker_mean_difference(xp, reps_p, dt):
    """(1/n) sum_i (x - x_i) in worker order (the all-reduce, reading above)."""
    acc = xp - np.asarray(reps_p[0], dtype=np.float32).astype(dt)
    for r in reps_p[1:]:
        acc = acc + (xp - np.asarray(r, dtype=np.float32).astype(dt))
    return acc / dt(len(reps_p))


def _global_adamw(x, m, v, replicas, *, gamma, eta, beta1, beta2, lam, eps, decay, t, dt):
    """Algorithm 7 (Appendix C): AdamW on the pseudo-gradient of round t."""
    if v is None:
        raise ValueError("Global AdamW needs the second-moment buffer v")
    b1, b2 = f32(beta1), f32(beta2)
    beta1_, beta2_ = dt(b1), dt(b2)
    one_minus_b1, one_minus_b2 = dt(1.0 - b1), dt(1.0 - b2)
    inv_gamma = dt(1.0 / f32(gamma))
    bc1 = dt(1.0 - beta_power(b1, t + 1))
    bc2 = dt(1.0 - beta_power(b2, t + 1))
    eta_, eps_, lam_ = dt(f32(eta)), dt(f32(eps)), dt(f32(lam))
    out = {"x": [], "m": [], "v": [], "u": [], "S": [], "delta": [], "B": None}
    for p in range(len(x)):
        xp = np.asarray(x[p], dtype=np.float32).astype(dt)
        mp = np.asarray(m[p], dtype=np.float32).astype(dt)
        vp = np.asarray(v[p], dtype=np.float32).astype(dt)
        delta = _worker_mean_difference(xp, [r[p] for r in replicas], dt)
        # Pseudo-gradient, momentum updates, bias corrections, parameter update.
        g = inv_gamma * delta
        m_new = beta1_ * mp + one_minus_b1 * g
        v_new = beta2_ * vp + one_minus_b2 * (g * g)
        m_hat = m_new / bc1
        v_hat = v_new / bc2
        lam_p = lam_ if decay[p] else dt(0.0)
        x_new = xp - eta_ * (m_hat / (np.sqrt(v_hat) + eps_) + lam_p * xp)
        out["x"].append(x_new)
        out["m"].append(m_new)
        out["v"].append(v_new)
        out["u"].append(g)
        out["S"].append(None)
        out["delta"].append(delta)
    return out


def synchronize(x, n):
    """Synchronisation step of Algorithm 1: every replica becomes x_{t+1,0}."""
    return [[np.array(a, dtype=np.float32, copy=True) for a in x] for _ in range(n)]


# --------------------------------------------------------------------------
# Algorithm 1 driver
# --------------------------------------------------------------------------

def _store(a):
    return np.asarray(a).astype(np.float32)


def init_state(x0, n, base):
    """Algorithm 1 initialisation: replicas = x_{0,0}, m_0 = 0, base state 0."""
    x = [_store(a) for a in x0]
    st = {
        "x": x,
        "m": [np.zeros_like(a) for a in x],
        "replicas": synchronize(x, n),
        "s1": [[np.zeros_like(a) for a in x] for _ in range(n)],
        "s2": [[np.zeros_like(a) for a in x] for _ in range(n)] if base == "adamw" else None,
        "base": base,
        "n": n,
    }
    return st


def local_steps(st, grads, *, H, lr, beta1, beta2=0.95, eps=1e-8, weight_decay=0.0,
                decay, first_step, prec="fp64"):
    """H local steps on every worker (inner loop of Algorithm 1), in place.

    grads(i, k) returns worker i's direction input for local step k (a list
    of per-tensor arrays).  first_step is the bias-correction count of the
    first of these steps.  State is stored as fp32 after every step.
    """
    n = st["n"]
    for i in range(n):
        for k in range(H):
            g = grads(i, k)
            for p in range(len(st["x"])):
                xr = st["replicas"][i][p]
                if st["base"] == "adamw":
                    wd = weight_decay if decay[p] else 0.0
                    xn, mn, vn = local_adamw_step(
                        xr, g[p], st["s1"][i][p], st["s2"][i][p], lr=lr, beta1=beta1,
                        beta2=beta2, eps=eps, weight_decay=wd, step=first_step + k,
                        prec=prec)
                    st["s2"][i][p] = _store(vn)
                else:
                    xn, mn = local_sgdm_step(xr, g[p], st["s1"][i][p], lr=lr,
                                             momentum=beta1, prec=prec)
                st["replicas"][i][p] = _store(xn)
                st["s1"][i][p] = _store(mn)
    return st


def communication_round(st, grads, t, *, H, local, glob, decay, prec="fp64"):
    """One outer iteration t of Algorithm 1, in place.

    local: dict of local hyperparameters (lr, beta1, beta2, eps, weight_decay).
    glob:  dict of global hyperparameters (eta, beta1, beta2, lam, mode, seed);
           the global step uses the local learning rate as gamma_t.
    The bias-correction count of local step k is s = t*H + k + 1.
    Returns the global-step output dict.
    """
    local_steps(st, grads, H=H, decay=decay, first_step=t * H + 1, prec=prec, **local)
    extra = {}
    if glob.get("rule", RULE_SIGN_MOMENTUM) == RULE_GLOBAL_ADAMW:
        extra["v"] = st.setdefault("v", [np.zeros_like(a) for a in st["x"]])
    res = global_step(st["x"], st["m"], st["replicas"], gamma=local["lr"], decay=decay,
                      t=t, prec=prec, **glob, **extra)
    st["x"] = [_store(a) for a in res["x"]]
    st["m"] = [_store(a) for a in res["m"]]
    if "v" in res:
        st["v"] = [_store(a) for a in res["v"]]
    st["replicas"] = synchronize(st["x"], st["n"])
    return res
