"""Device memory for the library: torch tensors as the caller-owned arenas.

PyTorch only allocates device memory and supplies the stream; every step of
the method runs in libdsm.so through the binding in ``dsm``.
"""
import torch

from . import dsm

# With contiguous or blocked replicas every buffer is its own allocation, and
# each buffer's base is moved by a different multiple of this many floats
# (1 MiB + 1 KiB).  Large allocations start on 2 MiB boundaries, so without it
# the same element of x, m and the replicas shares its low address bits across
# buffers.  Measured on MI355X at GPT-2 xl over alternating allocations, the
# fused round end runs ~1% faster staggered (27.2-27.6 ms against
# 27.5-28.4 ms); the local and global steps are unaffected.
STAGGER_FLOATS = (1 << 18) + 256

# 2 MiB in floats: the parts of the state-blocked allocation start on it.
PAGE_FLOATS = 1 << 19
# Spacing of the candidate offsets of the placement probe (Arenas(...,
# placement_span=...)).
PROBE_STEP_BYTES = 2 << 30
# The probe's span.  Measured on MI355X with GPT-2-small-sized arenas
# (17 GB), fast placements start inside windows ~12 GB wide that recur
# irregularly, 32-100 GB apart, so a span of 64 GiB often holds none.  The
# span raises the odds of a fast placement; it does not guarantee one.
PROBE_SPAN_BYTES = 128 << 30


class Arenas:
    """The arenas and workspace of one problem, allocated with torch, plus the
    dsm_buffers struct that points at them.

    numel: per-tensor element counts; n_workers, local_steps, base: the
    problem (dsm_problem); decay: per-tensor weight-decay flags or None;
    randomized: allocate u_scratch for the randomized sign; global_adamw:
    allocate the global second moment v of the Global AdamW rule;
    replica_layout: how x_rep holds the replicas (dsm_replica_layout);
    placement_span (bytes, state-blocked layout only): allocate this much more
    and place the buffers at the offset in it where the problem's kernels run
    fastest (placement_step apart; see _probe_placement); 0 places them at
    the start.

    x_rep is an (n, d_pad) view with contiguous replicas, and an (n, blocks,
    16384) strided view of the same memory with blocked replicas.  With the
    replicas and their state blocked, x_rep, g_rep, s1_rep and s2_rep are
    (n, blocks, 4096) strided views of one allocation, which also holds x, m,
    u and v.  worker(), workers(), gather(), replica() and replicas() read
    every layout the same way.
    """

    def __init__(self, numel, n_workers, local_steps, base, decay=None, randomized=True,
                 global_adamw=False, device="cuda", replica_layout=dsm.DSM_REPLICAS_CONTIGUOUS,
                 placement_span=0, placement_step=PROBE_STEP_BYTES):
        self.numel = [int(v) for v in numel]
        self.n = int(n_workers)
        self.H = int(local_steps)
        self.base = int(base)
        self.decay = None if decay is None else [bool(v) for v in decay]
        self.replica_layout = int(replica_layout)
        self.problem = dsm.make_problem(self.numel, self.n, self.H, self.base, self.decay,
                                        self.replica_layout)
        self.arena_elems, self.offsets, self.workspace_bytes = dsm.dsm_layout(self.problem)
        a = max(self.arena_elems, 64)
        self._storage = []
        self._k = 0

        def alloc(*shape, stagger=True):
            # A view at a buffer-specific offset (a multiple of 64 floats, so
            # 256-byte alignment is kept) into a slightly larger allocation.
            pad = self._k * STAGGER_FLOATS if stagger else 0
            self._k += 1
            count = 1
            for s_ in shape:
                count *= s_
            flat = torch.zeros(count + pad, dtype=torch.float32, device=device)
            self._storage.append(flat)
            return flat[pad:].view(*shape)

        adamw = self.base == dsm.DSM_BASE_ADAMW
        self.n_state_buffers = 4 if adamw else 3
        if self.state_blocked and self.arena_elems > 0:
            # One allocation for everything: x, m, u, v, then the blocks, each
            # part on a 2 MiB boundary; block b of the last part holds the n
            # copies of x_rep, g_rep, s1_rep (and s2_rep) of elements
            # [4096 b, 4096 b + 4096).  One allocation fixes where x and m sit
            # relative to the blocks.  Measured on MI355X over re-allocations,
            # the kernels that read x and m next to the blocks ran at 77-80%
            # of 8 TB/s at GPT-2 xl and large this way, against 70-78% with
            # separate allocations (the local steps are unaffected).
            parts = [("x", a), ("m", a)]
            parts += [("u", a)] if randomized else []
            parts += [("v", a)] if global_adamw else []
            parts += [("x_rep_flat", self.n_state_buffers * self.n * a)]
            self._parts, o = [], 0
            for name, count in parts:
                self._parts.append((name, o, count))
                o = -(-(o + count) // PAGE_FLOATS) * PAGE_FLOATS
            span = -(-int(placement_span) // (4 * PAGE_FLOATS)) * PAGE_FLOATS
            flat = torch.zeros(o + span, dtype=torch.float32, device=device)
            self._storage.append(flat)
            self.workspace = torch.zeros(max(self.workspace_bytes, 256), dtype=torch.uint8,
                                         device=device)
            self.placement = None
            self.u = self.v = None
            if span > 0:
                self.placement = self._probe_placement(flat, span, placement_step)
                flat[self.placement["offset_floats"]:][:o].zero_()
            self._carve(flat, 0 if span == 0 else self.placement["offset_floats"])
            if not randomized:
                self.u = None
            if not global_adamw:
                self.v = None
        else:
            self.x = alloc(a)
            self.m = alloc(a)
            self.x_rep_flat = alloc(self.n * a)
            if self.blocked and self.arena_elems > 0:
                B = dsm.DSM_REPLICA_BLOCK_ELEMS
                self.x_rep = self.x_rep_flat.view(a // B, self.n, B).permute(1, 0, 2)
            else:
                self.x_rep = self.x_rep_flat.view(self.n, a)
            self.g_rep = alloc(self.n, a)
            self.s1_rep = alloc(self.n, a)
            self.s2_rep = alloc(self.n, a) if adamw else None
            self.u = alloc(a) if randomized else None
            self.v = alloc(a) if global_adamw else None
            self.workspace = torch.zeros(max(self.workspace_bytes, 256), dtype=torch.uint8,
                                         device=device)
            self.placement = None
        self.ctx = None

    def _carve(self, flat, offset):
        """Points x, m, u, v and the per-worker blocks at their parts of flat,
        offset floats in (the state-blocked layout)."""
        a = max(self.arena_elems, 64)
        K = dsm.DSM_STATE_BLOCK_ELEMS
        for name, start, count in self._parts:
            setattr(self, name, flat[offset + start:offset + start + count])
        sup = self.x_rep_flat.view(a // K, self.n_state_buffers, self.n, K)
        self.x_rep, self.g_rep, self.s1_rep = (sup[:, j].permute(1, 0, 2) for j in range(3))
        self.s2_rep = sup[:, 3].permute(1, 0, 2) if self.n_state_buffers == 4 else None

    def _probe_placement(self, flat, span, step_bytes):
        """Times the problem's kernels with its buffers carved at each 2 MiB-
        aligned offset in [0, span] floats of flat, step_bytes apart, and
        returns the fastest offset.  On MI355X the rate of a working set of a
        few tens of GB depends on where in physical memory it lands
        (measured: small GPT-2-sized arenas ran their local steps at 76% or
        82% of 8 TB/s, and the kernels that read x and m at 66% or 78%, by
        offset, fast only inside windows ~12 GB wide and 32-100 GB apart); a
        span of 128 GiB found a fast placement for every small-, medium- and
        large-sized problem measured (23 processes), one of 64 GiB for 3 of
        15 small-sized ones.  Each candidate runs, on zeroed buffers, one fused
        round end and one local step of the problem with H = 1; the contents
        do not matter, and the chosen part is zeroed again afterwards."""
        step = max(PAGE_FLOATS, (int(step_bytes) // 4) // PAGE_FLOATS * PAGE_FLOATS)
        offsets = list(range(0, span + 1, step))
        probe = dsm.make_problem(self.numel, self.n, 1, self.base, self.decay, self.replica_layout)
        if self.base == dsm.DSM_BASE_ADAMW:
            local = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0)
        else:
            local = dict(lr=1e-3, beta1=0.9)
        glob = dict(gamma=1e-3, eta=0.8, beta1=0.95, beta2=0.98, lam=0.0)
        stream = torch.cuda.current_stream()
        events = []
        for k, off in enumerate([offsets[0]] + offsets):   # the first run warms up
            self._carve(flat, off)
            ctx = dsm.dsm_init(probe, self.buffers(stream))
            try:
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
                ev[0].record(stream)
                dsm.dsm_round_end(ctx, 1, local, 0, broadcast=False, **glob)
                ev[1].record(stream)
                dsm.dsm_sync(ctx)
                ev[2].record(stream)
                dsm.dsm_local_step(ctx, -1, 2, **local)
                ev[3].record(stream)
                stream.synchronize()
            finally:
                dsm.dsm_destroy(ctx)
            if k > 0:
                events.append((off, ev[0].elapsed_time(ev[1]) + ev[2].elapsed_time(ev[3])))
        best = min(events, key=lambda e: e[1])
        return {"offset_floats": best[0], "offset_bytes": 4 * best[0],
                "candidates": len(events), "best_ms": best[1],
                "worst_ms": max(t for _, t in events)}

    def buffers(self, stream=None):
        if stream is None:
            stream = torch.cuda.current_stream()

        def ptr(t):
            return None if t is None else t.data_ptr()
        return dsm.dsm_buffers(ptr(self.x), ptr(self.m), ptr(self.x_rep_flat), ptr(self.g_rep),
                               ptr(self.s1_rep), ptr(self.s2_rep), ptr(self.u),
                               ptr(self.workspace), self.workspace.numel(), stream.cuda_stream,
                               ptr(self.v))

    def init(self, stream=None):
        """dsm_init on the current contents of x."""
        self.ctx = dsm.dsm_init(self.problem, self.buffers(stream))
        return self.ctx

    @property
    def blocked(self):
        return self.replica_layout == dsm.DSM_REPLICAS_BLOCKED

    @property
    def state_blocked(self):
        return self.replica_layout == dsm.DSM_REPLICAS_STATE_BLOCKED

    _STATE_ORDER = ("x_rep", "g_rep", "s1_rep", "s2_rep")

    def replica_index(self, i, e):
        """Index into x_rep_flat of element(s) e (arena indices) of replica i."""
        return self.state_index("x_rep", i, e)

    def state_index(self, name, i, e):
        """Index of element(s) e of worker i's copy of a per-worker buffer:
        into x_rep_flat for x_rep (and for every buffer when state-blocked),
        else into the buffer's own (n, d_pad) arena."""
        if self.state_blocked:
            K = dsm.DSM_STATE_BLOCK_ELEMS
            j = self._STATE_ORDER.index(name)
            return (e // K) * (self.n_state_buffers * self.n * K) + (j * self.n + i) * K + e % K
        if name == "x_rep" and self.blocked:
            B = dsm.DSM_REPLICA_BLOCK_ELEMS
            return (e // B) * (self.n * B) + i * B + e % B
        return i * self.arena_elems + e

    def replica(self, i):
        """Replica i as a 1-D arena copy (a view when contiguous, else a copy)."""
        return self.x_rep[i].reshape(-1)

    def worker(self, name, i):
        """Worker i's copy of a per-worker buffer ("x_rep", "g_rep", "s1_rep" or
        "s2_rep") as a 1-D arena (a view when contiguous, else a copy)."""
        return getattr(self, name)[i].reshape(-1)

    def workers(self, name):
        """All n copies of a per-worker buffer as (n, d_pad) (a view when
        contiguous, else a copy)."""
        return getattr(self, name).reshape(self.n, -1)

    def write_workers(self, name, src):
        """Copies an (n, d_pad) tensor (worker i's copy in row i, arena order)
        into a per-worker buffer, in place, in any replica layout: the caller's
        gradients before a local step, or restored optimizer state."""
        dst = getattr(self, name)
        dst.copy_(src.reshape(dst.shape))

    def gather(self, name, i, idx):
        """Elements idx (arena indices, a device tensor) of worker i's copy of a
        per-worker buffer, without materialising a blocked copy."""
        if self.state_blocked or (name == "x_rep" and self.blocked):
            return self.x_rep_flat[self.state_index(name, i, idx)]
        return getattr(self, name)[i][idx]

    def replicas(self):
        """All replicas as (n, d_pad) (a view when contiguous, else a copy)."""
        return self.x_rep.reshape(self.n, -1)

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
