"""GPU path (libdsm.so through the C ABI) against the CPU oracle.

Seeded synthetic inputs at sizes the oracle finishes in seconds, spanning
several 16384-element chunks, ragged tensor ends (numel not a multiple of 4)
and an empty tensor.  Each call is compared element by element against the
oracle run from the same device state (copied to the host before the call),
to the bars described in tests/parity.py.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

from parity import (adamw_scales, det_flip_check, global_scales, rand_flip_check, rel_check, rms,
                    scaled_check, sgdm_scales)

pytestmark = pytest.mark.gpu

RAGGED = [1, 3, 4, 5, 63, 64, 65, 0, 1000, 16383, 16384, 16385, 40003]
DECAY = [i % 3 != 1 for i in range(len(RAGGED))]
# The layouts of dsm_problem.replica_layout.
LAYOUTS = [dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED, dsm.DSM_REPLICAS_STATE_BLOCKED]


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().copy()


def make(numel, n, H, base, decay=None, seed=0, randomized=True,
         layout=dsm.DSM_REPLICAS_CONTIGUOUS):
    ar = A.Arenas(numel, n, H, base, decay=decay, randomized=randomized, replica_layout=layout)
    gen = torch.Generator(device="cuda").manual_seed(seed)
    ar.x.normal_(0.0, 0.02, generator=gen)
    ar.init()
    return ar, gen


def per_tensor(ar, flat):
    """Host per-tensor arrays of one arena copy."""
    h = host(flat)
    return [h[o:o + n].copy() for o, n in zip(ar.offsets, ar.numel)]


def padding_mask(ar):
    mask = np.ones(ar.x.numel(), dtype=bool)
    for o, n in zip(ar.offsets, ar.numel):
        mask[o:o + n] = False
    return mask


# ---------------------------------------------------------------- Philox

@pytest.mark.parametrize("seed,tensor,t,q0,count", [
    (0, 0, 0, 0, 1000), (0x0123456789ABCDEF, 579, 12345, 77, 4099),
    ((1 << 64) - 1, 3, (1 << 32) - 1, (1 << 32) - 300, 300)])
def test_device_philox_matches_oracle(seed, tensor, t, q0, count):
    out = torch.zeros(4 * count, dtype=torch.int32, device="cuda")
    dsm.dsm_test_philox(seed, tensor, t, q0, count, out.data_ptr(),
                        torch.cuda.current_stream().cuda_stream)
    got = host(out).view(np.uint32).reshape(count, 4)
    q = np.arange(q0, q0 + count, dtype=np.uint64)
    want = np.stack(O.philox4x32_10(q, tensor, t, O.PHILOX_STREAM, seed & 0xFFFFFFFF, seed >> 32),
                    axis=1)
    np.testing.assert_array_equal(got, want)


# ---------------------------------------------------------------- local steps

def _randomize_state(ar, gen, adamw):
    """Arbitrary (non-zero) replica and base-optimizer state."""
    ar.x_rep.normal_(0.0, 0.02, generator=gen)
    ar.g_rep.normal_(0.0, 0.01, generator=gen)
    ar.s1_rep.normal_(0.0, 1e-3, generator=gen)
    if adamw:
        ar.s2_rep.normal_(0.0, 1e-3, generator=gen).square_()


@pytest.mark.parametrize("n,worker,step", [(3, -1, 1), (4, -1, 7), (4, 2, 3), (1, 0, 1000)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_local_adamw_parity(n, worker, step, layout):
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    ar, gen = make(RAGGED, n, 4, dsm.DSM_BASE_ADAMW, decay=DECAY, seed=n + step, layout=layout)
    _randomize_state(ar, gen, True)
    pad = padding_mask(ar)
    before = {k: [per_tensor(ar, ar.worker(k, i)) for i in range(n)]
              for k in ("x_rep", "g_rep", "s1_rep", "s2_rep")}
    pad_before = host(ar.replicas())[:, pad]
    dsm.dsm_local_step(ar.ctx, worker, step, **hp)
    after = {k: [per_tensor(ar, ar.worker(k, i)) for i in range(n)]
             for k in ("x_rep", "s1_rep", "s2_rep")}
    np.testing.assert_array_equal(host(ar.replicas())[:, pad], pad_before)
    nonbit = 0
    for i in range(n):
        for p in range(len(RAGGED)):
            x, g, m, v = (before[k][i][p] for k in ("x_rep", "g_rep", "s1_rep", "s2_rep"))
            gx, gm, gv = (after[k][i][p] for k in ("x_rep", "s1_rep", "s2_rep"))
            if worker not in (-1, i):
                for a, b in ((gx, x), (gm, m), (gv, v)):
                    np.testing.assert_array_equal(a, b)
                continue
            wd = hp["weight_decay"] if DECAY[p] else 0.0
            kw = dict(hp, weight_decay=wd, step=step)
            o32 = O.local_adamw_step(x, g, m, v, prec="fp32", **kw)
            o64 = O.local_adamw_step(x, g, m, v, prec="fp64", **kw)
            for name, gg, oo in (("x", gx, o32[0]), ("m", gm, o32[1]), ("v", gv, o32[2])):
                nonbit += rel_check(gg, oo, f"worker {i} tensor {p} {name}")
            s_m, s_v, s_x = adamw_scales(x, g, m, v, o64=o64, **kw)
            scaled_check(gx, o64[0], s_x, f"x vs fp64, worker {i} tensor {p}")
            scaled_check(gm, o64[1], s_m, f"m vs fp64, worker {i} tensor {p}")
            scaled_check(gv, o64[2], s_v, f"v vs fp64, worker {i} tensor {p}")
    print(f"adamw n={n} worker={worker}: {nonbit} elements not bit-identical to the fp32 oracle")
    assert nonbit == 0
    ar.destroy()


@pytest.mark.parametrize("n,worker", [(2, -1), (5, -1), (3, 0)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_local_sgdm_parity(n, worker, layout):
    hp = dict(lr=0.1, beta1=0.9)
    ar, gen = make(RAGGED, n, 2, dsm.DSM_BASE_SGD_MOMENTUM, seed=100 + n, layout=layout)
    _randomize_state(ar, gen, False)
    before = {k: [per_tensor(ar, ar.worker(k, i)) for i in range(n)]
              for k in ("x_rep", "g_rep", "s1_rep")}
    dsm.dsm_local_step(ar.ctx, worker, 1, **hp)
    after = {k: [per_tensor(ar, ar.worker(k, i)) for i in range(n)] for k in ("x_rep", "s1_rep")}
    nonbit = 0
    for i in range(n):
        for p in range(len(RAGGED)):
            x, g, m = (before[k][i][p] for k in ("x_rep", "g_rep", "s1_rep"))
            gx, gm = after["x_rep"][i][p], after["s1_rep"][i][p]
            if worker not in (-1, i):
                np.testing.assert_array_equal(gx, x)
                np.testing.assert_array_equal(gm, m)
                continue
            o32 = O.local_sgdm_step(x, g, m, lr=hp["lr"], momentum=hp["beta1"], prec="fp32")
            o64 = O.local_sgdm_step(x, g, m, lr=hp["lr"], momentum=hp["beta1"], prec="fp64")
            nonbit += rel_check(gx, o32[0], f"sgd x worker {i} tensor {p}")
            nonbit += rel_check(gm, o32[1], f"sgd m worker {i} tensor {p}")
            s_m, s_x = sgdm_scales(x, g, m, lr=hp["lr"], momentum=hp["beta1"])
            scaled_check(gx, o64[0], s_x, "sgd x vs fp64")
            scaled_check(gm, o64[1], s_m, "sgd m vs fp64")
    print(f"sgdm n={n}: {nonbit} elements not bit-identical to the fp32 oracle")
    assert nonbit == 0
    ar.destroy()


# ---------------------------------------------------------------- global step

def _ready_for_global(ar, gen, H, n):
    """H local SGD steps on every worker from perturbed replicas, then a
    random momentum, so the global step sees non-trivial x - x_i and m."""
    for _ in range(H):
        ar.g_rep.normal_(0.0, 1e-3, generator=gen)
        dsm.dsm_local_step(ar.ctx, -1, 1, lr=0.05, beta1=0.5)
    ar.m.normal_(0.0, 1.0, generator=gen)


GLOB = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)


@pytest.mark.parametrize("n,broadcast", [(1, True), (2, True), (3, True), (4, True), (4, False),
                                          (5, True), (8, True)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_global_det_parity(n, broadcast, layout):
    H = 2
    ar, gen = make(RAGGED, n, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, seed=200 + n,
                   layout=layout)
    _ready_for_global(ar, gen, H, n)
    x0, m0 = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
    reps = [per_tensor(ar, ar.replica(i)) for i in range(n)]
    rep_before = host(ar.replicas())
    dsm.dsm_global_step(ar.ctx, 5, mode=dsm.DSM_SIGN_DET, broadcast=broadcast, **GLOB)
    gx, gm = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
    o32 = O.global_step(x0, m0, reps, decay=DECAY, prec="fp32", **GLOB)
    o64 = O.global_step(x0, m0, reps, decay=DECAY, prec="fp64", **GLOB)
    nonbit, flips = 0, 0
    for p in range(len(RAGGED)):
        nonbit += rel_check(gx[p], o32["x"][p], f"x tensor {p}")
        nonbit += rel_check(gm[p], o32["m"][p], f"m tensor {p}")
        lam_p = GLOB["lam"] if DECAY[p] else 0.0
        s_u, s_m, s_x = global_scales(x0[p], m0[p], [r[p] for r in reps], o64["S"][p],
                                      lam_p=lam_p, **{k: v for k, v in GLOB.items() if k != "lam"})
        scaled_check(gm[p], o64["m"][p], s_m, f"m vs fp64 tensor {p}")
        # Sign decisions vs fp64: only where |u| is tiny.
        flip = o32["S"][p] != o64["S"][p]
        flips += det_flip_check(o32["S"][p], o64["S"][p], o64["u"][p], rms(o64["u"][p]),
                                f"tensor {p}")
        scaled_check(gx[p], o64["x"][p], s_x, f"x vs fp64 tensor {p}", mask=~flip)
    rep_after = host(ar.replicas())
    if broadcast:
        xa = host(ar.x)
        for i in range(n):
            for o, k in zip(ar.offsets, ar.numel):
                assert np.array_equal(rep_after[i, o:o + k].view(np.uint32),
                                      xa[o:o + k].view(np.uint32))
    else:
        # Replicas are left stale; the next local step reads the new x.
        np.testing.assert_array_equal(rep_after, rep_before)
        gx_now = per_tensor(ar, ar.x)
        m1 = [per_tensor(ar, ar.worker("s1_rep", i)) for i in range(n)]
        g1 = [per_tensor(ar, ar.worker("g_rep", i)) for i in range(n)]
        dsm.dsm_local_step(ar.ctx, -1, 1, lr=0.05, beta1=0.5)
        for i in range(n):
            xi = per_tensor(ar, ar.replica(i))
            for p in range(len(RAGGED)):
                ox, _ = O.local_sgdm_step(gx_now[p], g1[i][p], m1[i][p], lr=0.05, momentum=0.5,
                                          prec="fp32")
                assert np.array_equal(xi[p].view(np.uint32), ox.view(np.uint32)), (i, p)
        dsm.dsm_sync(ar.ctx)
        xa, ra = host(ar.x), host(ar.replicas())
        for i in range(n):
            for o, k in zip(ar.offsets, ar.numel):
                assert np.array_equal(ra[i, o:o + k].view(np.uint32), xa[o:o + k].view(np.uint32))
    print(f"global det n={n}: {nonbit} non-bit-identical vs fp32 oracle, {flips} sign flips vs fp64")
    assert nonbit == 0
    ar.destroy()


@pytest.mark.parametrize("n,mode,seed", [(2, dsm.DSM_SIGN_RAND_FLIP, 1),
                                         (4, dsm.DSM_SIGN_RAND_ZERO, (1 << 63) + 12345),
                                         (3, dsm.DSM_SIGN_RAND_FLIP, 2 ** 40 + 7),
                                         (8, dsm.DSM_SIGN_RAND_ZERO, 99)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_global_randomized_parity(n, mode, seed, layout):
    H = 1
    ar, gen = make(RAGGED, n, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, seed=300 + n,
                   layout=layout)
    _ready_for_global(ar, gen, H, n)
    x0, m0 = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
    reps = [per_tensor(ar, ar.replica(i)) for i in range(n)]
    t = 77
    dsm.dsm_global_step(ar.ctx, t, mode=mode, seed=seed, broadcast=True, **GLOB)
    gx, gm, gu = per_tensor(ar, ar.x), per_tensor(ar, ar.m), per_tensor(ar, ar.u)
    B = dsm.dsm_read_bounds(ar.ctx, len(RAGGED))
    o32 = O.global_step(x0, m0, reps, decay=DECAY, prec="fp32", t=t, mode=mode, seed=seed, **GLOB)
    o64 = O.global_step(x0, m0, reps, decay=DECAY, prec="fp64", t=t, mode=mode, seed=seed, **GLOB)
    nonbit = flips = 0
    for p in range(len(RAGGED)):
        assert B[p].view(np.uint32) == np.float32(o32["B"][p]).view(np.uint32), f"B tensor {p}"
        np.testing.assert_array_equal(gu[p].view(np.uint32), o32["u"][p].view(np.uint32))
        nonbit += rel_check(gm[p], o32["m"][p], f"m tensor {p}")
        nonbit += rel_check(gx[p], o32["x"][p], f"x tensor {p}")
        # fp64 side: u and m within the error bound, and every randomized
        # decision that differs from the fp64 oracle's (its own bound B_p =
        # max |u| in fp64, the same Philox words) lies inside the 1e-6 rms(u)
        # margin of Eq. (9) / Eq. (10).
        lam_p = GLOB["lam"] if DECAY[p] else 0.0
        s_u, s_m, s_x = global_scales(x0[p], m0[p], [r[p] for r in reps], o64["S"][p],
                                      lam_p=lam_p, **{k: v for k, v in GLOB.items() if k != "lam"})
        scaled_check(gu[p], o64["u"][p], s_u, f"u vs fp64 tensor {p}")
        scaled_check(gm[p], o64["m"][p], s_m, f"m vs fp64 tensor {p}")
        k = O.randomized_sign_uniforms(RAGGED[p], p, t, seed)
        flips += rand_flip_check(o32["S"][p], o64["S"][p], o64["u"][p], o64["B"][p], k, mode,
                                 rms(o64["u"][p]), f"tensor {p}")
        flip = o32["S"][p] != o64["S"][p]
        scaled_check(gx[p], o64["x"][p], s_x, f"x vs fp64 tensor {p}", mask=~flip)
    ra, xa = host(ar.replicas()), host(ar.x)
    for i in range(n):
        for o, k in zip(ar.offsets, ar.numel):
            assert np.array_equal(ra[i, o:o + k].view(np.uint32), xa[o:o + k].view(np.uint32))
    print(f"global rand n={n} mode={mode}: {nonbit} non-bit-identical vs fp32 oracle, "
          f"{flips} randomized decisions differ from fp64 (all inside the margin)")
    assert nonbit == 0
    ar.destroy()


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_bound_is_recomputed_when_it_shrinks(fused, layout):
    """B_p is max |u| of the current step only: after a step whose u is
    large, a step with u a thousand times smaller (smaller gradients, m reset
    to 0) gets the smaller bound, exactly, and the signs that go with it.  Split steps and fused round ends
    (H = 1, so the round end takes the only local step)."""
    n, H, mode, seed = 3, 1, dsm.DSM_SIGN_RAND_FLIP, 2024
    ar, gen = make(RAGGED, n, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, seed=77, layout=layout)
    local = dict(lr=0.05, beta1=0.0)   # no local momentum carries the large step over
    B_prev = None
    for t, scale in enumerate((1e3, 1.0)):
        ar.g_rep.normal_(0.0, 1e-3 * scale, generator=gen)
        if t > 0:
            ar.m.zero_()     # else beta1 m keeps u as large as before
        if fused:
            x0, m0 = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
            dsm.dsm_round_end(ar.ctx, t + 1, local, t, mode=mode, seed=seed, broadcast=True,
                              **GLOB)
            reps = None
        else:
            dsm.dsm_local_step(ar.ctx, -1, t + 1, **local)
            x0, m0 = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
            reps = [per_tensor(ar, ar.replica(i)) for i in range(n)]
            dsm.dsm_global_step(ar.ctx, t, mode=mode, seed=seed, broadcast=True, **GLOB)
        gx, gu = per_tensor(ar, ar.x), per_tensor(ar, ar.u)
        B = dsm.dsm_read_bounds(ar.ctx, len(RAGGED))
        for p in range(len(RAGGED)):
            want = np.float32(np.max(np.abs(gu[p]))) if gu[p].size else np.float32(0.0)
            assert B[p].view(np.uint32) == want.view(np.uint32), (t, p)
        if reps is not None:
            o32 = O.global_step(x0, m0, reps, decay=DECAY, prec="fp32", t=t, mode=mode, seed=seed,
                                **GLOB)
            for p in range(len(RAGGED)):
                assert B[p].view(np.uint32) == np.float32(o32["B"][p]).view(np.uint32)
                assert rel_check(gx[p], o32["x"][p], f"x tensor {p}, step {t}") == 0
        if B_prev is not None:
            nonempty = np.array([k > 0 for k in RAGGED])
            assert np.all(B[nonempty] < 1e-2 * B_prev[nonempty]), "the bound did not shrink"
        B_prev = B
    ar.destroy()


# ---------------------------------------------------------------- whole rounds

def test_tiny_rounds_free_running_bit_identical():
    """The tiny workload (8 x 2^17, n=4, H=4 AdamW, deterministic sign): three
    free-running rounds of Algorithm 1 on the GPU and in the fp32 oracle from
    the same inputs end bit-identical (no re-seeding between rounds)."""
    from paper_2411_17866_amd import workloads as W
    w = W.get("tiny")
    ar, gen = make(w.numel, w.n_workers, w.local_steps, w.base, decay=w.decay, seed=w.seed,
                   randomized=False)
    st = O.init_state(per_tensor(ar, ar.x), w.n_workers, "adamw")
    glob = dict(w.glob, mode=O.SIGN_DET, seed=0)
    for t in range(3):
        grads = {}
        for k in range(w.local_steps):
            for i in range(w.n_workers):
                W.fill_grads_(ar.g_rep[i], w, i, t * w.local_steps + k)
                grads[(i, k)] = per_tensor(ar, ar.worker("g_rep", i))
            dsm.dsm_local_step(ar.ctx, -1, t * w.local_steps + k + 1, **w.local)
        dsm.dsm_global_step(ar.ctx, t, gamma=w.local["lr"], mode=dsm.DSM_SIGN_DET,
                            broadcast=True, **w.glob)
        O.communication_round(st, lambda i, k: grads[(i, k)], t, H=w.local_steps, local=w.local,
                              glob=glob, decay=w.decay, prec="fp32")
        for p in range(len(w.numel)):
            for name, gpu, ora in (("x", per_tensor(ar, ar.x)[p], st["x"][p]),
                                   ("m", per_tensor(ar, ar.m)[p], st["m"][p])):
                assert np.array_equal(gpu.view(np.uint32), ora.view(np.uint32)), (t, name, p)
            for i in range(w.n_workers):
                assert np.array_equal(per_tensor(ar, ar.worker("s1_rep", i))[p], st["s1"][i][p])
                assert np.array_equal(per_tensor(ar, ar.worker("s2_rep", i))[p], st["s2"][i][p])
                assert np.array_equal(per_tensor(ar, ar.replica(i))[p], st["replicas"][i][p])
    ar.destroy()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_tiny_long_free_run_all_signs_and_paths(layout):
    """Twelve free-running rounds of the tiny workload, cycling the three
    signs and alternating the fused round end (lazy broadcast) with the split
    path (broadcast).  GPU and fp32 oracle start from the same inputs and are
    never re-seeded from each other; after every round x, m and every
    worker's AdamW state must be bit-identical."""
    from paper_2411_17866_amd import workloads as W
    w = W.get("tiny")
    H = w.local_steps
    ar, gen = make(w.numel, w.n_workers, H, w.base, decay=w.decay, seed=w.seed + 1,
                   layout=layout)
    st = O.init_state(per_tensor(ar, ar.x), w.n_workers, "adamw")
    modes = (dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP, dsm.DSM_SIGN_RAND_ZERO)
    seed = 0x5EED0000000D5
    for t in range(12):
        mode = modes[t % 3]
        fused = t % 2 == 1
        grads = {}
        for k in range(H):
            for i in range(w.n_workers):
                W.fill_grads_(ar.g_rep[i], w, i, t * H + k)
                grads[(i, k)] = per_tensor(ar, ar.worker("g_rep", i))
            s = t * H + k + 1
            if fused and k == H - 1:
                dsm.dsm_round_end(ar.ctx, s, w.local, t, gamma=w.local["lr"], mode=mode,
                                  seed=seed, broadcast=False, **w.glob)
            else:
                dsm.dsm_local_step(ar.ctx, -1, s, **w.local)
        if not fused:
            dsm.dsm_global_step(ar.ctx, t, gamma=w.local["lr"], mode=mode, seed=seed,
                                broadcast=True, **w.glob)
        O.communication_round(st, lambda i, k: grads[(i, k)], t, H=H, local=w.local,
                              glob=dict(w.glob, mode=mode, seed=seed), decay=w.decay,
                              prec="fp32")
        gx, gm = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
        for p in range(len(w.numel)):
            assert np.array_equal(gx[p].view(np.uint32), st["x"][p].view(np.uint32)), (t, "x", p)
            assert np.array_equal(gm[p].view(np.uint32), st["m"][p].view(np.uint32)), (t, "m", p)
        for i in range(w.n_workers):
            g1, g2 = per_tensor(ar, ar.worker("s1_rep", i)), per_tensor(ar, ar.worker("s2_rep", i))
            for p in range(len(w.numel)):
                assert np.array_equal(g1[p].view(np.uint32), st["s1"][i][p].view(np.uint32))
                assert np.array_equal(g2[p].view(np.uint32), st["s2"][i][p].view(np.uint32))
    ar.destroy()


def test_rerun_is_bitwise_deterministic():
    """Two identical runs (local steps, randomized global step) agree bit for bit."""
    outs = []
    for _ in range(2):
        ar, gen = make(RAGGED, 3, 2, dsm.DSM_BASE_ADAMW, decay=DECAY, seed=5)
        for k in range(2):
            ar.g_rep.normal_(0.0, 0.01, generator=gen)
            dsm.dsm_local_step(ar.ctx, -1, k + 1, lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8,
                               weight_decay=0.1)
        dsm.dsm_global_step(ar.ctx, 3, mode=dsm.DSM_SIGN_RAND_FLIP, seed=42, **GLOB)
        outs.append([host(t) for t in (ar.x, ar.m, ar.replicas(), ar.workers("s1_rep"), ar.workers("s2_rep"), ar.u)])
        ar.destroy()
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_state_machine_on_gpu():
    ar, gen = make([100, 5000], 2, 2, dsm.DSM_BASE_ADAMW, seed=9, randomized=False)
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_global_step(ar.ctx, 0, **GLOB)
    assert e.value.status == dsm.DSM_ERR_STATE
    dsm.dsm_local_step(ar.ctx, 0, 1, **hp)
    dsm.dsm_local_step(ar.ctx, 0, 2, **hp)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_local_step(ar.ctx, 0, 3, **hp)     # worker 0 past H
    assert e.value.status == dsm.DSM_ERR_STATE
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_global_step(ar.ctx, 0, **GLOB)     # worker 1 has 0 steps
    assert e.value.status == dsm.DSM_ERR_STATE
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_global_step(ar.ctx, 0, mode=dsm.DSM_SIGN_RAND_FLIP, **GLOB)  # no u_scratch
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG
    dsm.dsm_local_step(ar.ctx, 1, 1, **hp)
    dsm.dsm_local_step(ar.ctx, 1, 2, **hp)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_read_bounds(ar.ctx, 2)
    assert e.value.status == dsm.DSM_ERR_STATE
    for bad in (dict(GLOB, gamma=0.0), dict(GLOB, beta1=1.5), dict(GLOB, lam=-1.0)):
        with pytest.raises(dsm.DsmError) as e:
            dsm.dsm_global_step(ar.ctx, 0, **bad)
        assert e.value.status == dsm.DSM_ERR_INVALID_ARG
    with pytest.raises(dsm.DsmError):
        dsm.dsm_global_step(ar.ctx, 1 << 32, **GLOB)
    dsm.dsm_global_step(ar.ctx, 0, **GLOB)
    # dsm_sync restarts the round: local counts back to zero.
    dsm.dsm_local_step(ar.ctx, -1, 3, **hp)
    dsm.dsm_sync(ar.ctx)
    dsm.dsm_local_step(ar.ctx, -1, 3, **hp)
    dsm.dsm_local_step(ar.ctx, -1, 4, **hp)
    dsm.dsm_global_step(ar.ctx, 1, **GLOB)
    ar.destroy()


def test_read_bounds_checks_the_output_capacity():
    """dsm_read_bounds writes one float per tensor; an array with room for
    fewer is an argument error, not an overrun."""
    ar, gen = make(RAGGED, 2, 1, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, seed=8)
    ar.g_rep.normal_(0.0, 1e-3, generator=gen)
    dsm.dsm_local_step(ar.ctx, -1, 1, lr=0.05, beta1=0.5)
    dsm.dsm_global_step(ar.ctx, 0, mode=dsm.DSM_SIGN_RAND_FLIP, seed=1, **GLOB)
    with pytest.raises(dsm.DsmError) as e:
        dsm.dsm_read_bounds(ar.ctx, len(RAGGED) - 1)
    assert e.value.status == dsm.DSM_ERR_INVALID_ARG
    B = dsm.dsm_read_bounds(ar.ctx, len(RAGGED))
    assert B.shape == (len(RAGGED),) and np.all(B >= 0)
    ar.destroy()


def test_empty_problem_is_a_no_op():
    ar = A.Arenas([], 2, 1, dsm.DSM_BASE_ADAMW)
    ar.init()
    dsm.dsm_local_step(ar.ctx, -1, 1, lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8)
    dsm.dsm_global_step(ar.ctx, 0, mode=dsm.DSM_SIGN_RAND_FLIP, **GLOB)
    assert dsm.dsm_read_bounds(ar.ctx, 0).size == 0
    dsm.dsm_sync(ar.ctx)
    ar.destroy()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_only_empty_tensors_give_zero_bounds(layout):
    """Tensors that all have zero elements: no chunk to launch over, yet every
    tensor's bound is written (0), through the split and the fused paths."""
    ar = A.Arenas([0, 0, 0], 2, 2, dsm.DSM_BASE_SGD_MOMENTUM, replica_layout=layout)
    ar.init()
    dsm.dsm_local_step(ar.ctx, -1, 1, lr=0.05, beta1=0.9)
    dsm.dsm_local_step(ar.ctx, -1, 2, lr=0.05, beta1=0.9)
    dsm.dsm_global_step(ar.ctx, 0, mode=dsm.DSM_SIGN_RAND_FLIP, **GLOB)
    assert np.array_equal(dsm.dsm_read_bounds(ar.ctx, 3), np.zeros(3, np.float32))
    dsm.dsm_local_step(ar.ctx, -1, 3, lr=0.05, beta1=0.9)
    dsm.dsm_round_end(ar.ctx, 4, dict(lr=0.05, beta1=0.9), 1, mode=dsm.DSM_SIGN_RAND_ZERO,
                      broadcast=False, **GLOB)
    assert np.array_equal(dsm.dsm_read_bounds(ar.ctx, 3), np.zeros(3, np.float32))
    dsm.dsm_sync(ar.ctx)
    ar.destroy()


# ---------------------------------------------------------------- limits, degenerate cases

@pytest.mark.parametrize("layout", LAYOUTS)
def test_max_workers_every_entry_point(layout):
    """n = 64 (the largest worker count): local AdamW, deterministic and
    randomized global steps and the fused round end without broadcast, then a
    round whose first local step starts every worker from x, against the
    oracle."""
    n, H = 64, 2
    numel = [5, 1000, 16385]
    decay = [False, True, True]
    local = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    ar, gen = make(numel, n, H, dsm.DSM_BASE_ADAMW, decay=decay, seed=64, layout=layout)
    st = O.init_state(per_tensor(ar, ar.x), n, "adamw")
    for t, (mode, fused) in enumerate(((dsm.DSM_SIGN_DET, False), (dsm.DSM_SIGN_RAND_ZERO, False),
                                       (dsm.DSM_SIGN_RAND_FLIP, True), (dsm.DSM_SIGN_DET, False))):
        grads = {}
        for k in range(H):
            ar.g_rep.normal_(0.0, 0.01, generator=gen)
            for i in range(n):
                grads[(i, k)] = per_tensor(ar, ar.worker("g_rep", i))
            s = t * H + k + 1
            if fused and k == H - 1:
                dsm.dsm_round_end(ar.ctx, s, local, t, mode=mode, seed=3, broadcast=False, **GLOB)
            else:
                dsm.dsm_local_step(ar.ctx, -1, s, **local)
        if not fused:
            dsm.dsm_global_step(ar.ctx, t, mode=mode, seed=3, **GLOB)
        O.communication_round(st, lambda i, k: grads[(i, k)], t, H=H, local=local,
                              glob=dict({k: v for k, v in GLOB.items() if k != "gamma"},
                                        mode=mode, seed=3),
                              decay=decay, prec="fp32")
        gx, gm = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
        for p in range(len(numel)):
            assert np.array_equal(gx[p].view(np.uint32), st["x"][p].view(np.uint32)), (t, p)
            assert np.array_equal(gm[p].view(np.uint32), st["m"][p].view(np.uint32)), (t, p)
    ar.destroy()


@pytest.mark.parametrize("hp", [dict(eta=0.0, beta1=0.95, beta2=0.98, lam=0.1),
                                dict(eta=0.8, beta1=1.0, beta2=0.0, lam=0.0),
                                dict(eta=0.8, beta1=0.0, beta2=1.0, lam=0.0)])
def test_global_step_degenerate_hyperparameters(hp):
    """eta = 0 leaves x fixed; beta1 = 1 makes u the old momentum; beta2 = 1
    freezes the momentum; beta = 0 forgets it.  Against the oracle, bitwise."""
    n, H = 3, 1
    ar, gen = make(RAGGED, n, H, dsm.DSM_BASE_SGD_MOMENTUM, decay=DECAY, seed=77)
    _ready_for_global(ar, gen, H, n)
    x0, m0 = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
    reps = [per_tensor(ar, ar.replica(i)) for i in range(n)]
    dsm.dsm_global_step(ar.ctx, 0, gamma=1e-3, **hp)
    gx, gm = per_tensor(ar, ar.x), per_tensor(ar, ar.m)
    o32 = O.global_step(x0, m0, reps, gamma=1e-3, decay=DECAY, prec="fp32", **hp)
    for p in range(len(RAGGED)):
        assert np.array_equal(gx[p].view(np.uint32), o32["x"][p].view(np.uint32)), p
        assert np.array_equal(gm[p].view(np.uint32), o32["m"][p].view(np.uint32)), p
        if hp["eta"] == 0.0:
            assert np.array_equal(gx[p], x0[p])
        if hp["beta2"] == 1.0:
            assert np.array_equal(gm[p], m0[p])
    ar.destroy()
