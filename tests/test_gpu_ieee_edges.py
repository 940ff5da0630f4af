"""IEEE edge cases through the whole path, against the oracle: non-finite
gradients, and subnormal values (the build keeps denormals).

A diverging worker can hand the optimizer NaN or infinite gradients.  NaN,
+inf and -inf are planted in chosen gradient elements, including a ragged
tensor end and an element where every worker is infinite.  Two rounds then
run, each of H local steps and a global step with broadcast, for both bases
and all three signs.

Every output is compared with the fp32 oracle run from the same device
state.  NaN positions must agree, and every other value must be
bit-identical.  That covers the local states, x and m, and for the randomized
sign also u and the per-tensor bound B, which turns NaN or inf with its
tensor.  Section 3.1 defines the randomized sign only for a finite bound, so
a tensor whose B is NaN or inf must take a NaN step at every element, never a
finite step of a reversed (Eq. (9)) or zero (Eq. (10)) sign.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

NUMEL = [1, 3, 5, 64, 65, 1000, 16385, 40003]
DECAY = [i % 3 != 1 for i in range(len(NUMEL))]
N, H = 3, 2
# (round, local step) -> [(worker or None for every worker, tensor, element, value)]
PLANTS = {
    (0, 0): [(1, 5, 17, np.nan)],
    (0, 1): [(0, 6, 16384, np.inf)],
    (1, 0): [(2, 7, 20000, -np.inf), (0, 2, 4, np.nan)],
    (1, 1): [(None, 3, 10, np.inf)],
}
ADAM = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
SGD = dict(lr=0.05, beta1=0.9)
GLOB = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)
SEED = 0xC0FFEE


def tensors(ar, flat):
    torch.cuda.synchronize()
    h = flat.detach().cpu().numpy()
    return [h[o:o + k].copy() for o, k in zip(ar.offsets, ar.numel)]


def same(gpu, ora, what):
    g = np.asarray(gpu, dtype=np.float32)
    o = np.asarray(ora, dtype=np.float32)
    gn, on = np.isnan(g), np.isnan(o)
    assert np.array_equal(gn, on), f"{what}: NaN positions differ ({gn.sum()} vs {on.sum()})"
    bad = g[~gn].view(np.uint32) != o[~on].view(np.uint32)
    assert not bad.any(), f"{what}: {bad.sum()} finite-or-inf values differ"


def _set_grad(ar, i, e, val):
    """Element e (arena index) of worker i's gradient, in any layout."""
    if ar.state_blocked:
        ar.x_rep_flat[ar.state_index("g_rep", i, e)] = val
    else:
        ar.g_rep[i, e] = val


@pytest.mark.parametrize("mode", [dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP,
                                  dsm.DSM_SIGN_RAND_ZERO])
@pytest.mark.parametrize("base", [dsm.DSM_BASE_ADAMW, dsm.DSM_BASE_SGD_MOMENTUM])
@pytest.mark.parametrize("layout", [dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED,
                                    dsm.DSM_REPLICAS_STATE_BLOCKED])
def test_nonfinite_gradients_match_oracle(base, mode, layout):
    adamw = base == dsm.DSM_BASE_ADAMW
    local = ADAM if adamw else SGD
    ar = A.Arenas(NUMEL, N, H, base, decay=DECAY, randomized=True, replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(99 + 3 * base + mode)
    ar.x.normal_(0.0, 0.02, generator=gen)
    ar.init()
    keys = ("x_rep", "s1_rep") + (("s2_rep",) if adamw else ())
    seen_nan = seen_inf = False
    undefined_bounds = {"nan": 0, "inf": 0}
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        for t in range(2):
            for k in range(H):
                s = t * H + k + 1
                ar.g_rep.normal_(0.0, 1e-3, generator=gen)
                for w, p, j, val in PLANTS[(t, k)]:
                    for i in (range(N) if w is None else (w,)):
                        _set_grad(ar, i, ar.offsets[p] + j, float(val))
                before = {name: [tensors(ar, ar.worker(name, i)) for i in range(N)]
                          for name in keys + ("g_rep",)}
                dsm.dsm_local_step(ar.ctx, -1, s, **local)
                for i in range(N):
                    after = {name: tensors(ar, ar.worker(name, i)) for name in keys}
                    for p in range(len(NUMEL)):
                        args = [before[name][i][p] for name in ("x_rep", "g_rep", "s1_rep")]
                        if adamw:
                            kw = dict(ADAM, step=s)
                            kw["weight_decay"] = ADAM["weight_decay"] if DECAY[p] else 0.0
                            o = O.local_adamw_step(*args, before["s2_rep"][i][p], prec="fp32",
                                                   **kw)
                        else:
                            o = O.local_sgdm_step(*args, lr=SGD["lr"], momentum=SGD["beta1"],
                                                  prec="fp32")
                        for name, want in zip(keys, o):
                            same(after[name][p], want, f"t {t} k {k} worker {i} {name} tensor {p}")
            x0, m0 = tensors(ar, ar.x), tensors(ar, ar.m)
            reps = [tensors(ar, ar.replica(i)) for i in range(N)]
            dsm.dsm_global_step(ar.ctx, t, mode=mode, seed=SEED, broadcast=True, **GLOB)
            o = O.global_step(x0, m0, reps, decay=DECAY, t=t, mode=mode, seed=SEED, prec="fp32",
                              **GLOB)
            gx, gm = tensors(ar, ar.x), tensors(ar, ar.m)
            if mode != dsm.DSM_SIGN_DET:
                B = dsm.dsm_read_bounds(ar.ctx, len(NUMEL))
                gu = tensors(ar, ar.u)
            for p in range(len(NUMEL)):
                same(gx[p], o["x"][p], f"t {t} x tensor {p}")
                same(gm[p], o["m"][p], f"t {t} m tensor {p}")
                seen_nan |= bool(np.isnan(gx[p]).any() or np.isnan(gm[p]).any())
                seen_inf |= bool(np.isinf(gm[p]).any())
                if mode != dsm.DSM_SIGN_DET:
                    same(gu[p], o["u"][p], f"t {t} u tensor {p}")
                    same(B[p:p + 1], np.asarray([o["B"][p]], np.float32), f"t {t} B tensor {p}")
                    if not np.isfinite(B[p]):
                        assert np.all(np.isnan(gx[p])), \
                            f"t {t} tensor {p}: bound {B[p]} but a finite step was taken"
                        undefined_bounds["nan" if np.isnan(B[p]) else "inf"] += 1
            for i in range(N):
                for a, b in zip(ar.views(ar.replica(i)), ar.views(ar.x)):
                    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    # The planted values did reach the global state, and the randomized sign
    # met NaN bounds (and, for SGD, whose steps keep an infinite gradient
    # infinite, inf bounds).
    assert seen_nan and (seen_inf or adamw)
    if mode != dsm.DSM_SIGN_DET:
        assert undefined_bounds["nan"] > 0 and (undefined_bounds["inf"] > 0 or adamw), \
            undefined_bounds
    ar.destroy()


# Gradients down to the smallest subnormal.  Where one worker alone moves an
# element whose x is 0, the averaged difference and u of the global step end
# up subnormal, and the sign must still be +-1: a flushed denormal would make
# it 0.
TINY = [1e-36, 3e-38, 1e-39, 1e-40, 1e-41, 1e-42, 1e-43, 1e-44, 1.4e-45]
TINY_NUMEL = [1000, 64]
TINY_DECAY = [True, True]
MIN_NORMAL = np.float32(2.0 ** -126)
# gamma = 1 keeps (1 - beta1)/gamma small, so u stays subnormal for both bases.
GLOB_TINY = dict(GLOB, gamma=1.0)


@pytest.mark.parametrize("base", [dsm.DSM_BASE_ADAMW, dsm.DSM_BASE_SGD_MOMENTUM])
def test_subnormal_values_match_oracle(base):
    adamw = base == dsm.DSM_BASE_ADAMW
    local = ADAM if adamw else SGD
    nt = len(TINY)
    ar = A.Arenas(TINY_NUMEL, N, H, base, decay=TINY_DECAY, randomized=False)
    gen = torch.Generator(device="cuda").manual_seed(5 + base)
    ar.x.normal_(0.0, 0.02, generator=gen)
    o0, o1 = ar.offsets
    ar.x[o0:o0 + 2 * nt] = 0.0
    ar.x[o1:o1 + nt] = torch.tensor(TINY, dtype=torch.float32, device="cuda") * 100.0
    ar.x[o1 + nt:o1 + 2 * nt] = -torch.tensor(TINY, dtype=torch.float32, device="cuda")
    ar.init()
    keys = ("x_rep", "s1_rep") + (("s2_rep",) if adamw else ())
    subnormal_signs = 0
    tiny = torch.tensor(TINY, dtype=torch.float32, device="cuda")
    for t in range(2):
        for k in range(H):
            s = t * H + k + 1
            ar.g_rep.normal_(0.0, 1e-3, generator=gen)
            ar.g_rep[:, o0:o0 + 2 * nt] = 0.0
            ar.g_rep[0, o0:o0 + nt] = tiny              # one worker moves these
            ar.g_rep[:, o0 + nt:o0 + 2 * nt] = -tiny    # every worker moves these
            before = {name: [tensors_of(ar, ar.worker(name, i), TINY_NUMEL) for i in range(N)]
                      for name in keys + ("g_rep",)}
            dsm.dsm_local_step(ar.ctx, -1, s, **local)
            for i in range(N):
                after = {name: tensors_of(ar, ar.worker(name, i), TINY_NUMEL) for name in keys}
                for p in range(len(TINY_NUMEL)):
                    args = [before[name][i][p] for name in ("x_rep", "g_rep", "s1_rep")]
                    if adamw:
                        o = O.local_adamw_step(*args, before["s2_rep"][i][p], prec="fp32",
                                               **dict(ADAM, step=s))
                    else:
                        o = O.local_sgdm_step(*args, lr=SGD["lr"], momentum=SGD["beta1"],
                                              prec="fp32")
                    for name, want in zip(keys, o):
                        same(after[name][p], want, f"t {t} k {k} worker {i} {name} tensor {p}")
        x0, m0 = tensors_of(ar, ar.x, TINY_NUMEL), tensors_of(ar, ar.m, TINY_NUMEL)
        reps = [tensors_of(ar, ar.replica(i), TINY_NUMEL) for i in range(N)]
        dsm.dsm_global_step(ar.ctx, t, broadcast=True, **GLOB_TINY)
        o = O.global_step(x0, m0, reps, decay=TINY_DECAY, t=t, prec="fp32", **GLOB_TINY)
        gx, gm = tensors_of(ar, ar.x, TINY_NUMEL), tensors_of(ar, ar.m, TINY_NUMEL)
        for p in range(len(TINY_NUMEL)):
            same(gx[p], o["x"][p], f"t {t} x tensor {p}")
            same(gm[p], o["m"][p], f"t {t} m tensor {p}")
            u, S = o["u"][p], o["S"][p]
            subnormal_signs += int(np.sum((np.abs(u) > 0) & (np.abs(u) < MIN_NORMAL) & (S != 0)))
    # The case did reach subnormal momenta whose sign is +-1.
    assert subnormal_signs > 0
    ar.destroy()


def tensors_of(ar, flat, numel):
    torch.cuda.synchronize()
    h = flat.detach().cpu().numpy()
    return [h[o:o + k].copy() for o, k in zip(ar.offsets, numel)]
