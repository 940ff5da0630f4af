"""Device memory for the library: torch tensors as the caller-owned arenas.

PyTorch only allocates device memory and supplies the stream; every step of
the method runs in libdsm.so through the binding in ``dsm``.
"""
import torch

from . import dsm

# Each buffer's base is moved by a different multiple of this many floats
# (1 MiB + 1 KiB).  Large allocations start on 2 MiB boundaries, so without it
# the same element of x, m and the replicas shares its low address bits across
# buffers.  Measured on MI355X at GPT-2 xl over alternating allocations, the
# fused round end runs ~1% faster staggered (27.2-27.6 ms against
# 27.5-28.4 ms); the local and global steps are unaffected.
STAGGER_FLOATS = (1 << 18) + 256


class Arenas:
    """The arenas and workspace of one problem, allocated with torch, plus the
    dsm_buffers struct that points at them.

    numel: per-tensor element counts; n_workers, local_steps, base: the
    problem (dsm_problem); decay: per-tensor weight-decay flags or None;
    randomized: allocate u_scratch for the randomized sign; global_adamw:
    allocate the global second moment v of the Global AdamW rule.
    """

    def __init__(self, numel, n_workers, local_steps, base, decay=None, randomized=True,
                 global_adamw=False, device="cuda"):
        self.numel = [int(v) for v in numel]
        self.n = int(n_workers)
        self.H = int(local_steps)
        self.base = int(base)
        self.decay = None if decay is None else [bool(v) for v in decay]
        self.problem = dsm.make_problem(self.numel, self.n, self.H, self.base, self.decay)
        self.arena_elems, self.offsets, self.workspace_bytes = dsm.dsm_layout(self.problem)
        a = max(self.arena_elems, 64)
        self._storage = []
        self._k = 0

        def alloc(*shape):
            # A view at a buffer-specific offset (a multiple of 64 floats, so
            # 256-byte alignment is kept) into a slightly larger allocation.
            pad = self._k * STAGGER_FLOATS
            self._k += 1
            count = 1
            for s_ in shape:
                count *= s_
            flat = torch.zeros(count + pad, dtype=torch.float32, device=device)
            self._storage.append(flat)
            return flat[pad:].view(*shape)

        self.x = alloc(a)
        self.m = alloc(a)
        self.x_rep = alloc(self.n, a)
        self.g_rep = alloc(self.n, a)
        self.s1_rep = alloc(self.n, a)
        self.s2_rep = alloc(self.n, a) if self.base == dsm.DSM_BASE_ADAMW else None
        self.u = alloc(a) if randomized else None
        self.v = alloc(a) if global_adamw else None
        self.workspace = torch.zeros(max(self.workspace_bytes, 256), dtype=torch.uint8,
                                     device=device)
        self.ctx = None

    def buffers(self, stream=None):
        if stream is None:
            stream = torch.cuda.current_stream()

        def ptr(t):
            return None if t is None else t.data_ptr()
        return dsm.dsm_buffers(ptr(self.x), ptr(self.m), ptr(self.x_rep), ptr(self.g_rep),
                               ptr(self.s1_rep), ptr(self.s2_rep), ptr(self.u),
                               ptr(self.workspace), self.workspace.numel(), stream.cuda_stream,
                               ptr(self.v))

    def init(self, stream=None):
        """dsm_init on the current contents of x."""
        self.ctx = dsm.dsm_init(self.problem, self.buffers(stream))
        return self.ctx

    def views(self, flat):
        """Per-tensor views of one arena copy (a 1-D tensor of arena_elems)."""
        return [flat[o:o + n] for o, n in zip(self.offsets, self.numel)]

    def destroy(self):
        if self.ctx is not None:
            dsm.dsm_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass
