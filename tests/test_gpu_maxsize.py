"""Maximum sizes: one tensor of 2^32 + 53253 elements between two small ones.

Element offsets, chunk starts and replica strides then all need 64 bits, and
the randomized sign's Philox block counter j >> 2 passes 2^30.  Each base
optimizer runs two rounds:
  * a split round: dsm_local_step, then the randomized dsm_global_step with
    broadcast;
  * a fused round: dsm_round_end with the lazy broadcast, then dsm_sync.
Outputs are checked against the fp32 oracle on sampled elements:
  * around 2^31 and 2^32;
  * on chunk and piece seams;
  * on the ragged tail;
  * at random.
The two small tensors are checked whole.  The randomized bound B_p is checked
two ways: against the exact max |u| of each whole tensor, taken on the GPU;
and for the small tensors, against the oracle's own max.

AdamW runs with one worker (7 buffers, 120 GB); SGD with momentum runs with
two workers (9 buffers, 155 GB), whose second replica starts 2^32 elements
past the first; AdamW runs again with two workers and the replicas and their
state in 16 KiB blocks of one allocation (11 buffers, 189 GB).
"""
import gc

import numpy as np
import pytest
import torch

import oracle as O
from paper_2411_17866_amd import arena as A
from paper_2411_17866_amd import dsm

from parity import rel_check

pytestmark = pytest.mark.gpu

BIG = (1 << 32) + 3 * 16384 + 4101
NUMEL = [5, BIG, 7]
DECAY = [False, True, False]
GLOB = dict(eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)
SEED = 0x9E3779B97F4A7C15
CASES = {
    "adamw_n1": dict(base=dsm.DSM_BASE_ADAMW, n=1,
                     modes=(dsm.DSM_SIGN_RAND_FLIP, dsm.DSM_SIGN_DET),
                     local=dict(lr=2e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)),
    # Blocked replicas: the 64 KiB-block addressing past 2^32 elements.
    "sgdm_n2_blocked": dict(base=dsm.DSM_BASE_SGD_MOMENTUM, n=2,
                            modes=(dsm.DSM_SIGN_RAND_ZERO, dsm.DSM_SIGN_RAND_FLIP),
                            local=dict(lr=0.1, beta1=0.9), layout=dsm.DSM_REPLICAS_BLOCKED),
    # Replicas and their state in 16 KiB blocks: the block addressing and the
    # worker-interleaved local steps past 2^32 elements.
    "adamw_n2_state": dict(base=dsm.DSM_BASE_ADAMW, n=2,
                           modes=(dsm.DSM_SIGN_RAND_FLIP, dsm.DSM_SIGN_DET),
                           local=dict(lr=2e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
                           layout=dsm.DSM_REPLICAS_STATE_BLOCKED),
}


def _samples(rng, n_random=200_000):
    """(tensor index p, in-tensor index j) of the elements to check; the small
    tensors whole and in order, so the oracle can take their bound itself."""
    ps, js = [], []
    for p, k in enumerate(NUMEL):
        if k < 64:
            ps.append(np.full(k, p))
            js.append(np.arange(k))
    two31, two32 = 1 << 31, 1 << 32
    seams = two32 + 2048 * np.arange(0, 8 * 4 + 1)  # every piece of the chunks past 2^32
    edges = np.r_[np.arange(8), two31 + np.arange(-2, 2), two32 + np.arange(-2, 3),
                  seams - 1, seams, BIG - 8 + np.arange(8),
                  rng.integers(0, BIG, n_random, dtype=np.int64),
                  rng.integers(two32, BIG, 4000, dtype=np.int64)]
    edges = np.unique(edges[(edges >= 0) & (edges < BIG)])
    ps.append(np.full(edges.size, 1))
    js.append(edges)
    return np.concatenate(ps).astype(np.int64), np.concatenate(js).astype(np.int64)


class Big:
    def __init__(self, case):
        c = CASES[case]
        self.c = c
        self.n = c["n"]
        self.adamw = c["base"] == dsm.DSM_BASE_ADAMW
        self.ar = A.Arenas(NUMEL, self.n, 1, c["base"], decay=DECAY, randomized=True,
                           replica_layout=c.get("layout", dsm.DSM_REPLICAS_CONTIGUOUS))
        assert self.ar.arena_elems > (1 << 32)
        self.gen = torch.Generator(device="cuda").manual_seed(77 + self.n)
        self.ar.x.normal_(0.0, 0.02, generator=self.gen)
        self.ar.init()
        self.p, self.j = _samples(np.random.default_rng(5))
        self.idx = torch.as_tensor(np.asarray(self.ar.offsets)[self.p] + self.j, device="cuda")
        self.dec = np.asarray(DECAY)[self.p]
        self.state = ("x_rep", "g_rep", "s1_rep") + (("s2_rep",) if self.adamw else ())
        self.lr = c["local"]["lr"]

    def sample(self, flat):
        return flat[self.idx].cpu().numpy().copy()

    def sample_state(self, keys):
        torch.cuda.synchronize()
        return {k: [self.ar.gather(k, i, self.idx).cpu().numpy().copy() for i in range(self.n)]
                for k in keys}

    def local_oracle(self, before, i, s):
        """The oracle's local step s of worker i on the sampled elements."""
        names = ("x_rep", "s1_rep") + (("s2_rep",) if self.adamw else ())
        out = {k: np.empty(self.p.size, np.float32) for k in names}
        for dec in (True, False):
            sel = self.dec == dec
            if not sel.any():
                continue
            if self.adamw:
                kw = dict(self.c["local"], step=s)
                kw["weight_decay"] = kw["weight_decay"] if dec else 0.0
                res = O.local_adamw_step(*(before[k][i][sel] for k in self.state),
                                         prec="fp32", **kw)
            else:
                res = O.local_sgdm_step(*(before[k][i][sel] for k in self.state),
                                        lr=self.lr, momentum=self.c["local"]["beta1"],
                                        prec="fp32")
            for k, name in enumerate(names):
                out[name][sel] = res[k]
        return out

    def check_global(self, x0, m0, reps, t, mode):
        """x, m (and u, B when randomized) after a global step."""
        torch.cuda.synchronize()
        gx, gm = self.sample(self.ar.x), self.sample(self.ar.m)
        rand = mode != dsm.DSM_SIGN_DET
        if rand:
            B = dsm.dsm_read_bounds(self.ar.ctx, len(NUMEL))
            for q, uv in enumerate(self.ar.views(self.ar.u)):
                lo, hi = torch.aminmax(uv)
                exact = np.float32(max(hi.item(), -lo.item()))
                assert B[q].view(np.uint32) == exact.view(np.uint32), f"bound of tensor {q}"
            gu = self.sample(self.ar.u)
        nonbit = 0
        for q in range(len(NUMEL)):
            s_ = self.p == q
            whole = NUMEL[q] < 64
            kw = dict(gamma=self.lr, decay=[DECAY[q]], t=t, mode=mode, seed=SEED, prec="fp32",
                      tensor_ids=[q], **GLOB)
            if not whole:
                kw.update(element_ids=[self.j[s_]], bounds=[B[q]] if rand else None)
            o = O.global_step([x0[s_]], [m0[s_]], [[r[s_]] for r in reps], **kw)
            nonbit += rel_check(gx[s_], o["x"][0], f"t {t} x tensor {q}")
            nonbit += rel_check(gm[s_], o["m"][0], f"t {t} m tensor {q}")
            if rand:
                np.testing.assert_array_equal(gu[s_].view(np.uint32), o["u"][0].view(np.uint32))
                if whole:
                    assert np.float32(o["B"][0]).view(np.uint32) == B[q].view(np.uint32)
        return nonbit

    def close(self):
        """Free the arenas now (not when pytest drops the fixture value), so
        the next case's buffers never share the device with these."""
        self.ar.destroy()
        self.ar = self.idx = None
        gc.collect()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()

    def replicas_equal_x(self):
        torch.cuda.synchronize()
        for i in range(self.n):
            for a, b in zip(self.ar.views(self.ar.replica(i)), self.ar.views(self.ar.x)):
                assert torch.equal(a.view(torch.int32), b.view(torch.int32)), f"replica {i}"


@pytest.fixture(params=list(CASES))
def big(request):
    if torch.cuda.get_device_properties(0).total_memory < 200e9:
        pytest.skip("needs the full HBM of one MI355X")
    gc.collect()
    torch.cuda.empty_cache()
    b = Big(request.param)
    yield b
    b.close()


def test_max_size_split_then_fused_round(big):
    b, ar, c = big, big.ar, big.c
    glob = dict(gamma=b.lr, seed=SEED, **GLOB)
    nonbit = 0
    # Round t = 0: one local step, then the randomized global step with broadcast.
    ar.g_rep.normal_(0.0, 1e-3, generator=b.gen)
    before = b.sample_state(b.state)
    dsm.dsm_local_step(ar.ctx, -1, 1, **c["local"])
    after = b.sample_state([k for k in b.state if k != "g_rep"])
    for i in range(b.n):
        exp = b.local_oracle(before, i, 1)
        for name, want in exp.items():
            nonbit += rel_check(after[name][i], want, f"local worker {i} {name}")
    x0, m0 = b.sample(ar.x), b.sample(ar.m)
    dsm.dsm_global_step(ar.ctx, 0, mode=c["modes"][0], broadcast=True, **glob)
    nonbit += b.check_global(x0, m0, after["x_rep"], 0, c["modes"][0])
    b.replicas_equal_x()
    # Round t = 1: the fused round end (its only local step folded in), lazy
    # broadcast, then an explicit sync.
    ar.g_rep.normal_(0.0, 1e-3, generator=b.gen)
    before = b.sample_state(b.state)
    x0, m0 = b.sample(ar.x), b.sample(ar.m)
    dsm.dsm_round_end(ar.ctx, 2, c["local"], 1, mode=c["modes"][1], broadcast=False, **glob)
    after = b.sample_state(("s1_rep",) + (("s2_rep",) if b.adamw else ()))
    reps = []
    for i in range(b.n):
        exp = b.local_oracle(before, i, 2)
        for name in after:
            nonbit += rel_check(after[name][i], exp[name], f"fused worker {i} {name}")
        reps.append(exp["x_rep"])
    nonbit += b.check_global(x0, m0, reps, 1, c["modes"][1])
    dsm.dsm_sync(ar.ctx)
    b.replicas_equal_x()
    print(f"max size n={b.n}: {b.p.size} sampled elements, {nonbit} not bit-identical")
    assert nonbit == 0
