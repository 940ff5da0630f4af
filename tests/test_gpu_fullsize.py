"""Parity at full size: the GPT-2 1.5B-shaped workload (580 tensors,
d = 1,557,611,200, n = 4 replicas, H = 12 local AdamW steps) in the launch
configuration the benchmark times.

Every update is elementwise given the per-tensor bound, so outputs are
checked on sampled elements the oracle computes one by one (random elements
plus the first and last elements of every tensor and the chunk seams of the
largest one), against the oracle in fp32 and fp64 as in tests/parity.py.
The randomized bound B_p is checked against the maximum of |u| over the
whole tensor, computed independently on the GPU (exact), and against the
oracle on whole tensors for the smaller tensors.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm
from paper_2411_17866_amd import workloads as W

from parity import adamw_scales, global_scales, rel_check, rms, scaled_check

pytestmark = pytest.mark.gpu


def _sample_indices(ar, rng, n_random=200_000):
    """(tensor index p, element index j) pairs to check."""
    ps, js = [], []
    for p, k in enumerate(ar.numel):
        edge = np.unique(np.r_[np.arange(min(k, 8)), np.arange(max(k - 8, 0), k)])
        ps.append(np.full(edge.size, p))
        js.append(edge)
    big = int(np.argmax(ar.numel))
    seams = np.arange(16384, ar.numel[big], 16384 * 97)
    seams = np.unique(np.r_[seams - 1, seams])
    ps.append(np.full(seams.size, big))
    js.append(seams)
    sizes = np.asarray(ar.numel, dtype=np.float64)
    rp = rng.choice(len(ar.numel), size=n_random, p=sizes / sizes.sum())
    rj = (rng.random(n_random) * np.asarray(ar.numel)[rp]).astype(np.int64)
    ps.append(rp)
    js.append(rj)
    p = np.concatenate(ps).astype(np.int64)
    j = np.concatenate(js).astype(np.int64)
    return p, j


def _gather(flat, idx):
    return flat[idx].cpu().numpy().copy()


@pytest.fixture(scope="module")
def xl():
    w = W.get("xl")
    if torch.cuda.get_device_properties(0).total_memory < 200e9:
        pytest.skip("needs the full HBM of one MI355X")
    ar = A.Arenas(w.numel, w.n_workers, w.local_steps, w.base, decay=w.decay, randomized=True)
    gen = torch.Generator(device="cuda").manual_seed(w.seed)
    W.fill_params_(ar.x, w, gen)
    for i in range(w.n_workers):
        W.fill_grads_(ar.g_rep[i], w, i, 0)
    ar.init()
    rng = np.random.default_rng(2024)
    p, j = _sample_indices(ar, rng)
    idx = torch.as_tensor(np.asarray(ar.offsets)[p] + j, device="cuda")
    yield w, ar, p, j, idx
    ar.destroy()
    del ar
    torch.cuda.empty_cache()


def test_fullsize_local_adamw_sampled(xl):
    w, ar, p, j, idx = xl
    n = w.n_workers
    torch.cuda.synchronize()
    before = {k: [_gather(getattr(ar, k)[i], idx) for i in range(n)]
              for k in ("x_rep", "g_rep", "s1_rep", "s2_rep")}
    dsm.dsm_local_step(ar.ctx, -1, 1, **w.local)
    torch.cuda.synchronize()
    after = {k: [_gather(getattr(ar, k)[i], idx) for i in range(n)]
             for k in ("x_rep", "s1_rep", "s2_rep")}
    decay = np.asarray(w.decay)[p]
    nonbit = 0
    for i in range(n):
        for dec in (True, False):
            sel = decay == dec
            x, g, m, v = (before[k][i][sel] for k in ("x_rep", "g_rep", "s1_rep", "s2_rep"))
            kw = dict(w.local, weight_decay=w.local["weight_decay"] if dec else 0.0, step=1)
            o32 = O.local_adamw_step(x, g, m, v, prec="fp32", **kw)
            o64 = O.local_adamw_step(x, g, m, v, prec="fp64", **kw)
            got = [after[k][i][sel] for k in ("x_rep", "s1_rep", "s2_rep")]
            for name, gg, oo in zip("xmv", got, o32):
                nonbit += rel_check(gg, oo, f"xl worker {i} {name}")
            s_m, s_v, s_x = adamw_scales(x, g, m, v, o64=o64, **kw)
            for gg, oo, sc, name in zip(got, o64, (s_x, s_m, s_v), "xmv"):
                scaled_check(gg, oo, sc, f"xl worker {i} {name} vs fp64")
    print(f"xl local AdamW: {p.size} sampled elements x {n} workers, {nonbit} not bit-identical")


def _local_round(w, ar, t):
    """All H local steps of round t on every worker, fresh gradients per step,
    after restarting the round from the synchronised model."""
    dsm.dsm_sync(ar.ctx)
    for k in range(w.local_steps):
        s = t * w.local_steps + k + 1
        for i in range(w.n_workers):
            W.fill_grads_(ar.g_rep[i], w, i, s)
        dsm.dsm_local_step(ar.ctx, -1, s, **w.local)


def test_fullsize_global_det_sampled(xl):
    w, ar, p, j, idx = xl
    n = w.n_workers
    # Round 0 with its global step, then the local steps of round 1, so that
    # the global step under test sees a non-zero momentum.
    _local_round(w, ar, 0)
    dsm.dsm_global_step(ar.ctx, 0, gamma=w.local["lr"], **w.glob)
    _local_round(w, ar, 1)
    torch.cuda.synchronize()
    x0, m0 = _gather(ar.x, idx), _gather(ar.m, idx)
    reps = [_gather(ar.x_rep[i], idx) for i in range(n)]
    dsm.dsm_global_step(ar.ctx, 1, gamma=w.local["lr"], **w.glob)
    torch.cuda.synchronize()
    gx, gm = _gather(ar.x, idx), _gather(ar.m, idx)
    decay = np.asarray(w.decay)[p]
    nonbit = flips = 0
    for dec in (True, False):
        sel = decay == dec
        if not sel.any():
            continue
        args = dict(gamma=w.local["lr"], decay=[dec], **w.glob)
        o32 = O.global_step([x0[sel]], [m0[sel]], [[r[sel]] for r in reps], prec="fp32", **args)
        o64 = O.global_step([x0[sel]], [m0[sel]], [[r[sel]] for r in reps], prec="fp64", **args)
        nonbit += rel_check(gx[sel], o32["x"][0], f"xl global x decay={dec}")
        nonbit += rel_check(gm[sel], o32["m"][0], f"xl global m decay={dec}")
        lam_p = w.glob["lam"] if dec else 0.0
        s_u, s_m, s_x = global_scales(x0[sel], m0[sel], [r[sel] for r in reps], o64["S"][0],
                                      gamma=w.local["lr"], eta=w.glob["eta"],
                                      beta1=w.glob["beta1"], beta2=w.glob["beta2"], lam_p=lam_p)
        scaled_check(gm[sel], o64["m"][0], s_m, "xl global m vs fp64")
        flip = o32["S"][0] != o64["S"][0]
        if flip.any():
            assert np.all(np.abs(o64["u"][0][flip]) < 1e-6 * rms(o64["u"][0]))
        flips += int(flip.sum())
        scaled_check(gx[sel], o64["x"][0], s_x, "xl global x vs fp64", mask=~flip)
    # Broadcast: every replica equals x, checked on the GPU for the whole arena.
    for i in range(n):
        assert torch.equal(ar.x_rep[i].view(torch.int32), ar.x.view(torch.int32))
    print(f"xl global det: {p.size} sampled elements, {nonbit} not bit-identical, {flips} flips vs fp64")


def test_fullsize_global_randomized(xl):
    w, ar, p, j, idx = xl
    n = w.n_workers
    t, seed = 2, w.philox_seed
    _local_round(w, ar, t)
    torch.cuda.synchronize()
    whole = [q for q, (name, _) in enumerate(w.tensors)
             if name in ("wpe", "ln_f.weight", "ln_f.bias") or name.startswith("h0.")
             or name.startswith("h47.")]
    wx = [ar.views(ar.x)[q].cpu().numpy().copy() for q in whole]
    wm = [ar.views(ar.m)[q].cpu().numpy().copy() for q in whole]
    wr = [[ar.views(ar.x_rep[i])[q].cpu().numpy().copy() for q in whole] for i in range(n)]
    x0, m0 = _gather(ar.x, idx), _gather(ar.m, idx)
    reps = [_gather(ar.x_rep[i], idx) for i in range(n)]
    dsm.dsm_global_step(ar.ctx, t, gamma=w.local["lr"], mode=dsm.DSM_SIGN_RAND_FLIP, seed=seed,
                        **w.glob)
    B = dsm.dsm_read_bounds(ar.ctx, len(w.numel))
    # B_p is max |u| over each whole tensor: checked on the GPU from u_scratch
    # for every tensor (an exact maximum, computed independently by torch).
    u_views = ar.views(ar.u)
    Bt = torch.stack([uv.abs().max() for uv in u_views]).cpu().numpy()
    np.testing.assert_array_equal(B.view(np.uint32), Bt.view(np.uint32))
    # Whole tensors against the oracle: u and B bit-identical.
    gargs = dict(gamma=w.local["lr"], t=t, seed=seed, prec="fp32", **w.glob)
    ow = O.global_step(wx, wm, wr, decay=[w.decay[q] for q in whole], tensor_ids=whole,
                       mode=O.SIGN_RAND_FLIP, **gargs)
    for a, q in enumerate(whole):
        assert np.float32(ow["B"][a]).view(np.uint32) == B[q].view(np.uint32), w.tensors[q][0]
        np.testing.assert_array_equal(u_views[q].cpu().numpy().view(np.uint32),
                                      ow["u"][a].view(np.uint32))
        np.testing.assert_array_equal(ar.views(ar.x)[q].cpu().numpy().view(np.uint32),
                                      ow["x"][a].view(np.uint32))
    # Sampled elements of every tensor, with the tensor's bound from the GPU
    # (checked above) and each element's own Philox draw.
    torch.cuda.synchronize()
    gx, gm = _gather(ar.x, idx), _gather(ar.m, idx)
    qs = np.unique(p)
    sel = [p == q for q in qs]
    o = O.global_step([x0[s_] for s_ in sel], [m0[s_] for s_ in sel],
                      [[r[s_] for s_ in sel] for r in reps], decay=[w.decay[q] for q in qs],
                      tensor_ids=qs, element_ids=[j[s_] for s_ in sel],
                      bounds=[B[q] for q in qs], mode=O.SIGN_RAND_FLIP, **gargs)
    nonbit = 0
    for a, s_ in enumerate(sel):
        nonbit += rel_check(gm[s_], o["m"][a], f"xl rand m tensor {qs[a]}")
        nonbit += rel_check(gx[s_], o["x"][a], f"xl rand x tensor {qs[a]}")
    for i in range(n):
        assert torch.equal(ar.x_rep[i].view(torch.int32), ar.x.view(torch.int32))
    print(f"xl randomized: {len(whole)} whole tensors and {p.size} sampled elements, "
          f"{nonbit} not bit-identical")
