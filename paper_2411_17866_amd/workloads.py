"""Synthetic workloads: tensor shapes, hyperparameters and seeded inputs.

Holds none of the method's arithmetic.  The shapes are GPT-2 parameter sets
(the models of the paper's experiments, Section 4 and Table 1: small, medium,
large, plus the 1.5B "xl" shape), with the language-model head tied to the
token embedding.  Parameters are drawn from N(0, 0.02^2); worker gradients,
which stand in for the backward pass of a model on OpenWebText, are drawn
i.i.d. normal per (worker, local step) from seeded generators, optionally
with a heavy tail.  The oracle never imports this module; tests and the
benchmark feed the same generated tensors to both sides.
"""
from dataclasses import dataclass, field

VOCAB = 50257
CONTEXT = 1024

BASE_ADAMW = 0
BASE_SGD_MOMENTUM = 1


def gpt2_tensors(d_model, n_layer, vocab=VOCAB, context=CONTEXT):
    """(name, shape) of a GPT-2 parameter set in arena order."""
    d = d_model
    out = [("wte", (vocab, d)), ("wpe", (context, d))]
    for layer in range(n_layer):
        p = f"h{layer}."
        out += [
            (p + "ln_1.weight", (d,)), (p + "ln_1.bias", (d,)),
            (p + "attn.c_attn.weight", (d, 3 * d)), (p + "attn.c_attn.bias", (3 * d,)),
            (p + "attn.c_proj.weight", (d, d)), (p + "attn.c_proj.bias", (d,)),
            (p + "ln_2.weight", (d,)), (p + "ln_2.bias", (d,)),
            (p + "mlp.c_fc.weight", (d, 4 * d)), (p + "mlp.c_fc.bias", (4 * d,)),
            (p + "mlp.c_proj.weight", (4 * d, d)), (p + "mlp.c_proj.bias", (d,)),
        ]
    out += [("ln_f.weight", (d,)), ("ln_f.bias", (d,))]
    return out


def _numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


@dataclass
class Workload:
    name: str
    tensors: list                 # [(name, shape)]
    decay: list                   # weight decay applies (2-D tensors for GPT-2 shapes)
    n_workers: int
    local_steps: int
    base: int
    local: dict                   # lr, beta1, beta2, eps, weight_decay
    glob: dict                    # eta, beta1, beta2, lam
    sign_modes: tuple             # dsm_sign values this workload runs
    grad_sigma: float
    heavy_frac: float = 0.0       # fraction of gradient entries scaled by heavy_scale
    heavy_scale: float = 100.0
    param_sigma: float = 0.02
    seed: int = 0
    philox_seed: int = 0x5EED5EED2411
    notes: str = field(default="")

    @property
    def numel(self):
        return [_numel(s) for _, s in self.tensors]

    @property
    def d(self):
        return sum(self.numel)


# Global step of every workload: the Lion-recommended beta1 0.95, beta2 0.98,
# lambda 0.1 the paper uses (Section 4, implementations) and eta 0.8, a value
# in each of its tuning grids.
GLOBAL = dict(eta=0.8, beta1=0.95, beta2=0.98, lam=0.1)


def _gpt2(name, d_model, n_layer, **kw):
    tensors = gpt2_tensors(d_model, n_layer)
    return Workload(name=name, tensors=tensors, decay=[len(s) == 2 for _, s in tensors],
                    glob=dict(GLOBAL), **kw)


def get(name):
    """The named workload: tiny, small, medium, large or xl."""
    if name == "tiny":
        tensors = [(f"t{i}", (1 << 17,)) for i in range(8)]
        return Workload(name="tiny", tensors=tensors, decay=[True] * 8, n_workers=4,
                        local_steps=4, base=BASE_ADAMW,
                        local=dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
                        glob=dict(GLOBAL), sign_modes=(0,), grad_sigma=0.01, seed=11)
    if name == "small":
        return _gpt2("small", 768, 12, n_workers=8, local_steps=12, base=BASE_ADAMW,
                     local=dict(lr=5e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
                     sign_modes=(0,), grad_sigma=1e-3, seed=12)
    if name == "medium":
        return _gpt2("medium", 1024, 24, n_workers=8, local_steps=12, base=BASE_SGD_MOMENTUM,
                     local=dict(lr=0.1, beta1=0.9, beta2=0.0, eps=0.0, weight_decay=0.0),
                     sign_modes=(1,), grad_sigma=1e-3, seed=13)
    if name == "large":
        return _gpt2("large", 1280, 36, n_workers=8, local_steps=24, base=BASE_ADAMW,
                     local=dict(lr=2e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
                     sign_modes=(0,), grad_sigma=1e-3, heavy_frac=0.01, seed=14)
    if name == "xl":
        return _gpt2("xl", 1600, 48, n_workers=4, local_steps=12, base=BASE_ADAMW,
                     local=dict(lr=2e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
                     sign_modes=(0, 1), grad_sigma=1e-3, seed=15)
    raise KeyError(f"unknown workload {name!r}")


NAMES = ("tiny", "small", "medium", "large", "xl")


def grad_seed(w, worker, step):
    """Seed of worker `worker`'s gradient at local step `step` (global count)."""
    return (w.seed * 1_000_003 + worker * 10_007 + step * 131 + 7) % (2 ** 63)


def fill_params_(x, w, generator):
    """x ~ N(0, param_sigma^2), in place (a torch tensor on any device)."""
    x.normal_(0.0, w.param_sigma, generator=generator)
    return x


def fill_grads_(g, w, worker, step):
    """g ~ N(0, grad_sigma^2) with an optional heavy tail, in place, seeded by
    (workload seed, worker, step).  g is a torch tensor on any device."""
    import torch
    gen = torch.Generator(device=g.device)
    gen.manual_seed(grad_seed(w, worker, step))
    g.normal_(0.0, w.grad_sigma, generator=gen)
    if w.heavy_frac > 0:
        mask = torch.rand(g.shape, generator=gen, device=g.device) < w.heavy_frac
        g.mul_(torch.where(mask, w.heavy_scale, 1.0).to(g.dtype))
    return g
