"""Parity at full size for every GPT-2-shaped workload, in the launch
configuration the benchmark times:

  small   124M parameters, n = 8, H = 12, AdamW, deterministic sign
  medium  355M, n = 8, H = 12, SGD + Polyak momentum, randomized sign Eq. (9)
  large   774M, n = 8, H = 24, AdamW, heavy-tailed gradients, deterministic
  xl      1.56B, n = 4, H = 12, AdamW, deterministic and randomized sign

each with contiguous replicas, with 64 KiB-blocked replicas, and with the
replicas and their state in 16 KiB blocks of one allocation (the benchmark's
layout).
Every update is elementwise given the per-tensor bound, so outputs are
checked on sampled elements the oracle computes one by one (random elements,
the first and last elements of every tensor, chunk seams of the largest
one), against the oracle in fp32 and fp64 as in tests/parity.py.  Each
workload runs one local step (sampled), split rounds ending in
dsm_global_step, and a fused round ending in dsm_round_end (sampled).  The
randomized bound B_p is checked against the exact max |u| of every whole
tensor on the GPU, and against the oracle on whole tensors for a subset.
"""
import gc

import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm
from paper_2411_17866_amd import workloads as W

from parity import (adamw_scales, det_flip_check, global_scales, rand_flip_check, rel_check,
                    rms, scaled_check, sgdm_scales)

pytestmark = pytest.mark.gpu


def _sample_indices(ar, rng, n_random=150_000):
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
    return np.concatenate(ps).astype(np.int64), np.concatenate(js).astype(np.int64)


def _gather(flat, idx):
    return flat[idx].cpu().numpy().copy()


class Run:
    """One workload's arenas, initialised, plus the sampled elements."""

    def __init__(self, name, layout):
        self.w = W.get(name)
        w = self.w
        self.adamw = w.base == W.BASE_ADAMW
        self.mode = dsm.DSM_SIGN_RAND_FLIP if 1 in w.sign_modes else dsm.DSM_SIGN_DET
        # As the bench places them: state-blocked arenas under 120 GB at the
        # probed offset of a 128 GiB larger allocation.
        working_set = 4 * w.d * (4 + (4 if self.adamw else 3) * w.n_workers)
        probe = layout == dsm.DSM_REPLICAS_STATE_BLOCKED and working_set < 120e9
        self.ar = A.Arenas(w.numel, w.n_workers, w.local_steps, w.base, decay=w.decay,
                           randomized=True, global_adamw=True, replica_layout=layout,
                           placement_span=A.PROBE_SPAN_BYTES if probe else 0)
        assert (self.ar.placement is not None) == probe
        gen = torch.Generator(device="cuda").manual_seed(w.seed)
        W.fill_params_(self.ar.x, w, gen)
        self.ar.init()
        rng = np.random.default_rng(2024)
        self.p, self.j = _sample_indices(self.ar, rng)
        self.idx = torch.as_tensor(np.asarray(self.ar.offsets)[self.p] + self.j, device="cuda")
        self.decay = np.asarray(w.decay)[self.p]
        self.state_keys = ("x_rep", "g_rep", "s1_rep") + (("s2_rep",) if self.adamw else ())

    def grads(self, s):
        for i in range(self.w.n_workers):
            W.fill_grads_(self.ar.g_rep[i], self.w, i, s)

    def local(self, s):
        dsm.dsm_local_step(self.ar.ctx, -1, s, **self.w.local)

    def sample_state(self, keys):
        torch.cuda.synchronize()
        return {k: [self.ar.gather(k, i, self.idx).cpu().numpy().copy()
                    for i in range(self.w.n_workers)] for k in keys}

    def glob_kw(self):
        return dict(gamma=self.w.local["lr"], seed=self.w.philox_seed, **self.w.glob)


LAYOUT_NAMES = {dsm.DSM_REPLICAS_CONTIGUOUS: "contiguous", dsm.DSM_REPLICAS_BLOCKED: "blocked",
                dsm.DSM_REPLICAS_STATE_BLOCKED: "state-blocked"}
CASES = [(wl, lay) for lay in (dsm.DSM_REPLICAS_CONTIGUOUS, dsm.DSM_REPLICAS_BLOCKED)
         for wl in ("small", "medium", "large", "xl")]
# The bench's layout and placement for every GPT-2 size: the replicas and
# their state blocked, and below xl carved at the probed offset.
CASES += [(wl, dsm.DSM_REPLICAS_STATE_BLOCKED) for wl in ("small", "medium", "large", "xl")]


@pytest.fixture(scope="module", params=CASES,
                ids=[f"{wl}-{LAYOUT_NAMES[lay]}" for wl, lay in CASES])
def run(request):
    if torch.cuda.get_device_properties(0).total_memory < 200e9:
        pytest.skip("needs the full HBM of one MI355X")
    gc.collect()
    torch.cuda.empty_cache()
    r = Run(*request.param)
    yield r
    # Free the arenas now, not when pytest drops the fixture value, so the next
    # workload (or module) never shares the device with them.
    r.ar.destroy()
    r.ar = r.idx = None
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _local_oracle(r, before, i, sel, s, dec, prec):
    """Oracle local step of worker i on the sampled elements sel."""
    w = r.w
    if r.adamw:
        kw = dict(w.local, weight_decay=w.local["weight_decay"] if dec else 0.0, step=s)
        return O.local_adamw_step(*(before[k][i][sel] for k in ("x_rep", "g_rep", "s1_rep",
                                                                "s2_rep")), prec=prec, **kw)
    return O.local_sgdm_step(*(before[k][i][sel] for k in ("x_rep", "g_rep", "s1_rep")),
                             lr=w.local["lr"], momentum=w.local["beta1"], prec=prec)


def test_fullsize_local_step_sampled(run):
    r = run
    w = r.w
    r.grads(1)
    before = r.sample_state(r.state_keys)
    r.local(1)
    after = r.sample_state([k for k in r.state_keys if k != "g_rep"])
    nonbit = 0
    for i in range(w.n_workers):
        for dec in (True, False):
            sel = r.decay == dec
            if not sel.any():
                continue
            o32 = _local_oracle(r, before, i, sel, 1, dec, "fp32")
            o64 = _local_oracle(r, before, i, sel, 1, dec, "fp64")
            x, g, m = (before[k][i][sel] for k in ("x_rep", "g_rep", "s1_rep"))
            if r.adamw:
                kw = dict(w.local, weight_decay=w.local["weight_decay"] if dec else 0.0, step=1)
                s_m, s_v, s_x = adamw_scales(x, g, m, before["s2_rep"][i][sel], o64=o64, **kw)
                names, scales = ("x_rep", "s1_rep", "s2_rep"), (s_x, s_m, s_v)
            else:
                s_m, s_x = sgdm_scales(x, g, m, lr=w.local["lr"], momentum=w.local["beta1"])
                names, scales = ("x_rep", "s1_rep"), (s_x, s_m)
            for k, name in enumerate(names):
                got = after[name][i][sel]
                nonbit += rel_check(got, o32[k], f"{w.name} worker {i} {name}")
                scaled_check(got, o64[k], scales[k], f"{w.name} worker {i} {name} vs fp64")
    print(f"{w.name} local step: {r.p.size} sampled elements x {w.n_workers} workers, "
          f"{nonbit} not bit-identical")
    assert nonbit == 0


def _check_global_sampled(r, x0, m0, reps, t, gx, gm, mode):
    """Sampled x, m after a global step against the oracle (randomized: with
    each tensor's bound from the GPU, checked separately)."""
    w = r.w
    kw = dict(gamma=w.local["lr"], t=t, seed=w.philox_seed, **w.glob)
    nonbit = flips = 0
    if mode == dsm.DSM_SIGN_DET:
        for dec in (True, False):
            s_ = r.decay == dec
            if not s_.any():
                continue
            args = ([x0[s_]], [m0[s_]], [[rp[s_]] for rp in reps])
            o32 = O.global_step(*args, decay=[dec], prec="fp32", **kw)
            o64 = O.global_step(*args, decay=[dec], prec="fp64", **kw)
            nonbit += rel_check(gx[s_], o32["x"][0], f"{w.name} global x")
            nonbit += rel_check(gm[s_], o32["m"][0], f"{w.name} global m")
            lam_p = w.glob["lam"] if dec else 0.0
            _, s_m, s_x = global_scales(x0[s_], m0[s_], [rp[s_] for rp in reps], o64["S"][0],
                                        gamma=w.local["lr"], eta=w.glob["eta"],
                                        beta1=w.glob["beta1"], beta2=w.glob["beta2"], lam_p=lam_p)
            scaled_check(gm[s_], o64["m"][0], s_m, f"{w.name} global m vs fp64")
            flip = o32["S"][0] != o64["S"][0]
            flips += det_flip_check(o32["S"][0], o64["S"][0], o64["u"][0], rms(o64["u"][0]),
                                    f"{w.name} global sign")
            scaled_check(gx[s_], o64["x"][0], s_x, f"{w.name} global x vs fp64", mask=~flip)
        return nonbit, flips
    # Randomized: each tensor's bound is the GPU's B_p (checked separately
    # against the exact max |u| of the whole tensor).  The fp64 side evaluates
    # u in fp64 on the same elements and decides with that bound and the same
    # Philox words; rms_p(u) for the flip margin is estimated from the
    # tensor's sampled elements.
    B = dsm.dsm_read_bounds(r.ar.ctx, len(w.numel))
    qs = np.unique(r.p)
    sel = [r.p == q for q in qs]
    args = ([x0[s_] for s_ in sel], [m0[s_] for s_ in sel], [[rp[s_] for s_ in sel] for rp in reps])
    okw = dict(decay=[w.decay[q] for q in qs], tensor_ids=qs, element_ids=[r.j[s_] for s_ in sel],
               bounds=[B[q] for q in qs], mode=mode, **kw)
    o = O.global_step(*args, prec="fp32", **okw)
    o64 = O.global_step(*args, prec="fp64", **okw)
    for a, s_ in enumerate(sel):
        q = qs[a]
        nonbit += rel_check(gm[s_], o["m"][a], f"{w.name} rand m tensor {q}")
        nonbit += rel_check(gx[s_], o["x"][a], f"{w.name} rand x tensor {q}")
        k = O.randomized_sign_uniforms_at(r.j[s_], int(q), t, w.philox_seed)
        flips += rand_flip_check(o["S"][a], o64["S"][a], o64["u"][a], float(B[q]), k, mode,
                                 rms(o64["u"][a]), f"{w.name} rand sign tensor {q}")
    return nonbit, flips


def _whole_subset(r):
    return [q for q, (name, _) in enumerate(r.w.tensors)
            if name in ("wpe", "ln_f.weight", "ln_f.bias") or name.startswith("h0.")]


def _check_bounds(r, t, whole, wx, wm, wr, mode):
    """B_p = max |u| over every whole tensor (on the GPU, exact), and the
    oracle's u and B on the whole tensors of the subset."""
    w, ar = r.w, r.ar
    B = dsm.dsm_read_bounds(ar.ctx, len(w.numel))
    u_views = ar.views(ar.u)
    Bt = torch.stack([uv.abs().max() for uv in u_views]).cpu().numpy()
    np.testing.assert_array_equal(B.view(np.uint32), Bt.view(np.uint32))
    okw = dict(gamma=w.local["lr"], decay=[w.decay[q] for q in whole], t=t, seed=w.philox_seed,
               tensor_ids=whole, mode=mode, **w.glob)
    ow = O.global_step(wx, wm, wr, prec="fp32", **okw)
    ow64 = O.global_step(wx, wm, wr, prec="fp64", **okw)
    flips = 0
    for a, q in enumerate(whole):
        assert np.float32(ow["B"][a]).view(np.uint32) == B[q].view(np.uint32), w.tensors[q][0]
        np.testing.assert_array_equal(u_views[q].cpu().numpy().view(np.uint32),
                                      ow["u"][a].view(np.uint32))
        # Whole tensors: the fp64 oracle's own bound max |u| and the exact rms.
        k = O.randomized_sign_uniforms(w.numel[q], q, t, w.philox_seed)
        flips += rand_flip_check(ow["S"][a], ow64["S"][a], ow64["u"][a], ow64["B"][a], k, mode,
                                 rms(ow64["u"][a]), f"{w.name} whole {w.tensors[q][0]}")
    return flips


def test_fullsize_split_rounds_sampled(run):
    r = run
    w, ar = r.w, r.ar
    H = w.local_steps
    nonbit = flips = whole_flips = 0
    # Round t = 1 sees a non-zero momentum.  A workload with both signs runs the
    # deterministic one in round t = 0 and the randomized one in round t = 1.
    modes = (dsm.DSM_SIGN_DET, r.mode) if 0 in w.sign_modes else (r.mode, r.mode)
    for t in (0, 1):
        mode = modes[t]
        dsm.dsm_sync(ar.ctx)
        for k in range(H):
            r.grads(t * H + k + 1)
            r.local(t * H + k + 1)
        torch.cuda.synchronize()
        x0, m0 = _gather(ar.x, r.idx), _gather(ar.m, r.idx)
        reps = [ar.gather("x_rep", i, r.idx).cpu().numpy().copy() for i in range(w.n_workers)]
        whole = _whole_subset(r)
        if mode != dsm.DSM_SIGN_DET:
            wx = [ar.views(ar.x)[q].cpu().numpy().copy() for q in whole]
            wm = [ar.views(ar.m)[q].cpu().numpy().copy() for q in whole]
            wr = []
            for i in range(w.n_workers):
                rep_views = ar.views(ar.replica(i))
                wr.append([rep_views[q].cpu().numpy().copy() for q in whole])
                del rep_views
        dsm.dsm_global_step(ar.ctx, t, mode=mode, **r.glob_kw())
        torch.cuda.synchronize()
        if mode != dsm.DSM_SIGN_DET:
            whole_flips += _check_bounds(r, t, whole, wx, wm, wr, mode)
        gx, gm = _gather(ar.x, r.idx), _gather(ar.m, r.idx)
        nb, fl = _check_global_sampled(r, x0, m0, reps, t, gx, gm, mode)
        nonbit += nb
        flips += fl
        for i in range(w.n_workers):
            for a, b in zip(ar.views(ar.replica(i)), ar.views(ar.x)):
                assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    print(f"{w.name} split rounds: {r.p.size} sampled elements, {nonbit} not bit-identical, "
          f"{flips} sign decisions differ from fp64 on the samples, {whole_flips} on the whole "
          f"tensors of the subset (each inside its 1e-6 rms(u) margin)")
    assert nonbit == 0


def test_fullsize_fused_round_sampled(run):
    """H-1 local steps, then dsm_round_end with the lazy broadcast; the
    oracle recomputes step H from the sampled step-(H-1) state."""
    r = run
    w, ar = r.w, r.ar
    H = w.local_steps
    t = 2
    dsm.dsm_sync(ar.ctx)
    for k in range(H - 1):
        r.grads(t * H + k + 1)
        r.local(t * H + k + 1)
    r.grads(t * H + H)
    before = r.sample_state(r.state_keys)
    x0, m0 = _gather(ar.x, r.idx), _gather(ar.m, r.idx)
    dsm.dsm_round_end(ar.ctx, t * H + H, w.local, t, mode=r.mode, broadcast=False, **r.glob_kw())
    after = r.sample_state(("s1_rep",) + (("s2_rep",) if r.adamw else ()))
    gx, gm = _gather(ar.x, r.idx), _gather(ar.m, r.idx)
    nonbit = 0
    reps = []
    for i in range(w.n_workers):
        xr = np.empty_like(x0)
        for dec in (True, False):
            sel = r.decay == dec
            if not sel.any():
                continue
            o = _local_oracle(r, before, i, sel, t * H + H, dec, "fp32")
            nonbit += rel_check(after["s1_rep"][i][sel], o[1], f"{w.name} fused s1")
            if r.adamw:
                nonbit += rel_check(after["s2_rep"][i][sel], o[2], f"{w.name} fused s2")
            xr[sel] = o[0]
        reps.append(xr.astype(np.float32))
    nb, flips = _check_global_sampled(r, x0, m0, reps, t, gx, gm, r.mode)
    print(f"{w.name} fused round: {r.p.size} sampled elements, {nonbit + nb} not bit-identical, "
          f"{flips} sign decisions differ from fp64 (each inside its 1e-6 rms(u) margin)")
    assert nonbit + nb == 0


def test_fullsize_first_step_after_lazy_round_end(run):
    """A fused round that ends without broadcast leaves every replica stale,
    so the next local step of all workers reads x once in one launch.  Each
    worker's step is checked against the oracle's step from x."""
    r = run
    w, ar = r.w, r.ar
    H = w.local_steps
    t = 3
    dsm.dsm_sync(ar.ctx)
    for k in range(H - 1):
        r.grads(t * H + k + 1)
        r.local(t * H + k + 1)
    r.grads(t * H + H)
    dsm.dsm_round_end(ar.ctx, t * H + H, w.local, t, mode=r.mode, broadcast=False, **r.glob_kw())
    s = (t + 1) * H + 1
    r.grads(s)
    before = r.sample_state(r.state_keys)
    x0 = _gather(ar.x, r.idx)
    r.local(s)
    after = r.sample_state([k for k in r.state_keys if k != "g_rep"])
    nonbit = 0
    for i in range(w.n_workers):
        start = dict(before)
        start["x_rep"] = [x0] * w.n_workers      # a stale replica's step starts from x
        for dec in (True, False):
            sel = r.decay == dec
            if not sel.any():
                continue
            o = _local_oracle(r, start, i, sel, s, dec, "fp32")
            names = ("x_rep", "s1_rep") + (("s2_rep",) if r.adamw else ())
            for k, name in enumerate(names):
                nonbit += rel_check(after[name][i][sel], o[k], f"{w.name} from-x worker {i} {name}")
    print(f"{w.name} first step after a lazy round end: {r.p.size} sampled elements x "
          f"{w.n_workers} workers, {nonbit} not bit-identical")
    assert nonbit == 0


VARIANT_RULES = {dsm.DSM_RULE_LOOKAHEAD: O.RULE_LOOKAHEAD,
                 dsm.DSM_RULE_SIGNED_SLOWMO: O.RULE_SIGNED_SLOWMO,
                 dsm.DSM_RULE_GLOBAL_ADAMW: O.RULE_GLOBAL_ADAMW}
# Global AdamW (Algorithm 7) takes its own learning rate eta and epsilon.
ADAMW_GLOB = dict(eta=1e-3, beta1=0.9, beta2=0.95, lam=0.1, eps=1e-8)


XL_CASES = [c for c in CASES if c[0] == "xl"]


@pytest.mark.parametrize("run", XL_CASES, indirect=True,
                         ids=[f"xl-{LAYOUT_NAMES[lay]}" for _, lay in XL_CASES])
def test_fullsize_global_variants_sampled(run):
    """Lookahead, signed SlowMo (Section 4.1) and Global AdamW (Algorithm 7) at
    the xl size, each after H local steps, against the oracle on the sampled
    elements: x, m (and v) bit for bit against fp32; x against fp64 within the
    error bound, signed SlowMo's sign decisions allowed to differ only where
    the averaged difference is below 1e-6 of its rms."""
    r = run
    w, ar = r.w, r.ar
    H = w.local_steps
    nonbit = 0
    for k_rule, (rule, orule) in enumerate(VARIANT_RULES.items()):
        t = 5 + k_rule
        dsm.dsm_sync(ar.ctx)
        for k in range(H):
            r.grads(t * H + k + 1)
            r.local(t * H + k + 1)
        torch.cuda.synchronize()
        adamw = rule == dsm.DSM_RULE_GLOBAL_ADAMW
        glob = ADAMW_GLOB if adamw else w.glob
        x0, m0 = _gather(ar.x, r.idx), _gather(ar.m, r.idx)
        v0 = _gather(ar.v, r.idx) if adamw else None
        reps = [ar.gather("x_rep", i, r.idx).cpu().numpy().copy() for i in range(w.n_workers)]
        dsm.dsm_global_step(ar.ctx, t, rule=rule, gamma=w.local["lr"], **glob)
        torch.cuda.synchronize()
        gx, gm = _gather(ar.x, r.idx), _gather(ar.m, r.idx)
        gv = _gather(ar.v, r.idx) if adamw else None
        kw = dict(gamma=w.local["lr"], t=t, rule=orule, **glob)
        for dec in (True, False):
            s_ = r.decay == dec
            if not s_.any():
                continue
            args = ([x0[s_]], [m0[s_]], [[rp[s_]] for rp in reps])
            vkw = dict(v=[v0[s_]]) if adamw else {}
            o32 = O.global_step(*args, decay=[dec], prec="fp32", **kw, **vkw)
            o64 = O.global_step(*args, decay=[dec], prec="fp64", **kw, **vkw)
            nonbit += rel_check(gx[s_], o32["x"][0], f"{w.name} rule {rule} x")
            nonbit += rel_check(gm[s_], o32["m"][0], f"{w.name} rule {rule} m")
            if adamw:
                nonbit += rel_check(gv[s_], o32["v"][0], f"{w.name} rule {rule} v")
            ok = np.ones(int(s_.sum()), dtype=bool)
            if rule == dsm.DSM_RULE_SIGNED_SLOWMO:
                flip = np.sign(o32["delta"][0]) != np.sign(o64["delta"][0])
                if flip.any():
                    assert np.all(np.abs(o64["delta"][0][flip]) < 1e-6 * rms(o64["delta"][0]))
                ok &= ~flip
            err = np.abs(gx[s_].astype(np.float64) - o64["x"][0])
            step = O.f32(glob["eta"]) * (1.0 if adamw else O.f32(w.local["lr"]))
            if adamw:
                # x moves by eta * r with r = m_hat / (sqrt(v_hat) + eps), which can
                # be large where the pseudo-gradient is small against m; and the
                # worker sum that forms it cancels, so its fp32 relative error is
                # up to the condition number kappa = mean_i |x - x_i| / |Delta|.
                # Elements with Delta = 0 in fp64 have no finite bound.
                lam_p = O.f32(glob["lam"]) if dec else 0.0
                x064 = x0[s_].astype(np.float64)
                r64 = (x064 - o64["x"][0]) / O.f32(glob["eta"]) - lam_p * x064
                spread = np.mean([np.abs(x064 - rp[s_]) for rp in reps], axis=0)
                d64 = np.abs(o64["delta"][0])
                ok &= d64 > 0
                kappa = np.where(d64 > 0, spread / np.where(d64 > 0, d64, 1.0), 0.0)
                mag = np.abs(r64) * (1.0 + kappa) + np.abs(o64["m"][0]) + 1.0
            else:
                mag = np.abs(o64["u"][0]) + np.abs(o64["m"][0]) + 1.0
            bound = 64 * 2.0 ** -24 * (np.abs(o64["x"][0]) + np.abs(x0[s_]) + step * mag)
            bad = ok & (err > bound)
            if bad.any():
                k = int(np.argmax(np.where(ok, err / bound, 0.0)))
                raise AssertionError(
                    f"{w.name} rule {rule} x vs fp64: {int(bad.sum())} elements over the bound; "
                    f"worst: x0 {x0[s_][k]!r} m0 {m0[s_][k]!r} v0 {None if v0 is None else v0[s_][k]!r} "
                    f"reps {[rp[s_][k] for rp in reps]} gpu x {gx[s_][k]!r} fp32 x {o32['x'][0][k]!r} "
                    f"fp64 x {o64['x'][0][k]!r} u {o64['u'][0][k]!r} m {o64['m'][0][k]!r} "
                    f"err {err[k]:.3e} bound {bound[k]:.3e}")
        for i in range(w.n_workers):
            for a, b in zip(ar.views(ar.replica(i)), ar.views(ar.x)):
                assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    print(f"{w.name} Lookahead, signed SlowMo and Global AdamW: {r.p.size} sampled elements, "
          f"{nonbit} not bit-identical")
    assert nonbit == 0

