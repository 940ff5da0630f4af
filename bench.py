"""Benchmark of the distributed sign momentum hot path on one MI355X.

One step = one outer iteration of Algorithm 1 on the GPT-2 1.5B-shaped
workload (580 fp32 tensors, d = 1,557,611,200), n = 4 worker replicas:
H = 12 fused local AdamW steps over all replicas, then one fused global step
(worker average, sign momentum, decoupled weight decay, broadcast).  Every
input is resident in HBM before timing starts.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload xl] [--sign det|rand]
                    [--path fused|split] [--replica-layout blocked|contiguous]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "param-updates/s and achieved HBM GB/s (% peak) for local step + global sign step"
BYTES_LOCAL_ADAMW = 28     # x, g, m, v read; x, m, v written (fp32)
BYTES_LOCAL_SGDM = 20      # x, g, m read; x, m written


def bytes_global(n, randomized):
    # x, m, n replicas read; x, m, n replicas written; the randomized sign
    # adds the u round trip (write in pass 1, read in pass 2) and reads x twice.
    return 16 + 8 * n + (12 if randomized else 0)


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("dsm_kernels.hip", "philox_device.h", "dsm_internal.h"):
        with open(os.path.join(ROOT, "paper_2411_17866_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel_hash, workload, name):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when the counters were taken on a different kernel source, another
    workload, or do not cover the kernel."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_hash:
        return None
    k = rec.get("kernels", {}).get(name)
    return None if k is None else k.get("bytes_per_launch")


def _oracle_round_time(O, w, x0, grads, decay, prec):
    """Seconds the oracle takes for one round of Algorithm 1 (n workers, H
    local steps, deterministic global step) on the given whole tensors."""
    base = "adamw" if w.base == 0 else "sgd"
    st = O.init_state(x0, w.n_workers, base)
    t0 = time.perf_counter()
    O.communication_round(st, lambda i, k: grads[i], 0, H=w.local_steps, local=w.local,
                          glob=dict(w.glob, mode=O.SIGN_DET, seed=0), decay=decay, prec=prec)
    return time.perf_counter() - t0


def cpu_baseline(w, ar):
    """The oracle as it stands (numpy, one host thread) on bounded samples of
    the same workload: one round of Algorithm 1 over whole tensors, in fp64
    (its accuracy mode) and in fp32 (the GPU path's arithmetic type).  The
    samples cover every tensor shape class: fp64 runs on wpe, ln_f and
    transformer layer 0, fp32 on wpe, ln_f and the last layer (each about
    32M parameters at xl).  Every update is elementwise, so the rates carry
    over to the whole workload (extrapolated, labelled so)."""
    import numpy as np
    import torch

    import oracle as O

    names = [name for name, _ in w.tensors]
    last = max((int(nm[1:].split(".")[0]) for nm in names if nm.startswith("h")), default=None)
    subsets = {"fp64": ("h0.", "wpe", "ln_f."),
               "fp32": (f"h{last}." if last is not None else "h0.", "wpe", "ln_f.")}
    torch.cuda.synchronize()
    out = {"unit": "param-updates/s", "cores": 1, "kind": "oracle",
           "host_threads_available": len(os.sched_getaffinity(0))}
    for prec, prefixes in subsets.items():
        idx = [i for i, nm in enumerate(names) if nm.startswith(prefixes)]
        if not idx:                       # a workload with no GPT-2 names: all of it
            idx = list(range(len(names)))

        def take(flat):
            return [flat[ar.offsets[i]:ar.offsets[i] + ar.numel[i]].cpu().numpy() for i in idx]
        x0 = take(ar.x)
        elems = torch.cat([torch.arange(ar.offsets[i], ar.offsets[i] + ar.numel[i], device="cuda")
                           for i in idx])
        bounds = np.cumsum([0] + [ar.numel[i] for i in idx])
        grads = []
        for k in range(w.n_workers):
            gk = ar.gather("g_rep", k, elems).cpu().numpy()
            grads.append([gk[bounds[a]:bounds[a + 1]] for a in range(len(idx))])
        del elems
        d_s = int(sum(ar.numel[i] for i in idx))
        dt = _oracle_round_time(O, w, x0, grads, [w.decay[i] for i in idx], prec)
        updates = w.n_workers * w.local_steps * d_s + d_s
        out[prec] = {"value": updates / dt, "seconds": dt, "parameters": d_s,
                     "tensors": ", ".join(sorted({names[i].split(".")[0] for i in idx})),
                     "full_step_seconds_extrapolated":
                         (w.n_workers * w.local_steps + 1) * w.d / (updates / dt)}
    out["value"] = out["fp32"]["value"]
    out["sample"] = (f"one round (n={w.n_workers}, H={w.local_steps} local steps + deterministic "
                     f"global step) of the oracle on whole tensors, one host thread: fp32 on "
                     f"{out['fp32']['tensors']} ({out['fp32']['parameters']} of {w.d} parameters, "
                     f"{out['fp32']['seconds']:.1f} s), fp64 on {out['fp64']['tensors']} "
                     f"({out['fp64']['parameters']} parameters, {out['fp64']['seconds']:.1f} s); "
                     f"value is the fp32 rate")
    return out


def _sample_elements(ar, rng, n_random):
    """(tensor p, in-tensor index j) pairs: the first and last four elements of
    every tensor plus random ones spread by size."""
    import numpy as np
    ps, js = [], []
    for p, k in enumerate(ar.numel):
        if k == 0:
            continue
        e = np.unique(np.r_[np.arange(min(k, 4)), np.arange(max(k - 4, 0), k)])
        ps.append(np.full(e.size, p))
        js.append(e)
    sizes = np.asarray(ar.numel, dtype=np.float64)
    rp = rng.choice(len(ar.numel), size=n_random, p=sizes / sizes.sum())
    rj = (rng.random(n_random) * sizes[rp]).astype(np.int64)
    p = np.concatenate(ps + [rp]).astype(np.int64)
    j = np.concatenate(js + [rj]).astype(np.int64)
    key = np.unique(np.asarray(ar.offsets)[p] + j, return_index=True)[1]
    return p[key], j[key]


def parity_check(w, ar, run_round, t, mode, first_step, n_random=150_000):
    """One more round of the timed path, untimed, checked against the oracle on
    sampled elements: x and m, and every worker's base-optimizer state, bit for
    bit against the fp32 oracle (Algorithm 1 with Algorithm 2/3 as the base);
    the sign decisions of the global step against the fp64 oracle evaluated on
    the same fp32 inputs, where a flip is allowed only inside the 1e-6 rms(u)
    margin (Eq. (7), and Eqs. (9)/(10) for the randomized sign).  Every update
    is elementwise given each tensor's bound, so sampled elements are exact;
    the randomized sign takes each tensor's bound from the device."""
    import numpy as np
    import torch

    import oracle as O
    from paper_2411_17866_amd import dsm

    n = w.n_workers
    adamw = w.base == 0
    p, j = _sample_elements(ar, np.random.default_rng(2411), n_random)
    idx = torch.as_tensor(np.asarray(ar.offsets)[p] + j, device="cuda")
    g = lambda t_: t_[idx].cpu().numpy().copy()
    torch.cuda.synchronize()
    gw = lambda name, i: ar.gather(name, i, idx).cpu().numpy().copy()
    x0, m0 = g(ar.x), g(ar.m)
    s1 = [gw("s1_rep", i) for i in range(n)]
    s2 = [gw("s2_rep", i) for i in range(n)] if adamw else None
    grads = [gw("g_rep", i) for i in range(n)]
    run_round()
    torch.cuda.synchronize()
    got = {"x": g(ar.x), "m": g(ar.m)}
    for i in range(n):
        got[f"s1[{i}]"] = gw("s1_rep", i)
        if adamw:
            got[f"s2[{i}]"] = gw("s2_rep", i)
    B = dsm.dsm_read_bounds(ar.ctx, len(ar.numel)) if mode != dsm.DSM_SIGN_DET else None
    # The round's local steps, from the replicas equal to x (fresh after a
    # broadcast, or stale and read as x after a lazy round end).
    dec = np.asarray(w.decay)[p]
    reps = [x0.copy() for _ in range(n)]
    want = {}
    for i in range(n):
        xi, mi, vi = reps[i], s1[i], (s2[i] if adamw else None)
        for k in range(w.local_steps):
            for d_ in (True, False):
                sel = dec == d_
                if adamw:
                    lw = dict(w.local, weight_decay=w.local["weight_decay"] if d_ else 0.0)
                    a, b, c = O.local_adamw_step(xi[sel], grads[i][sel], mi[sel], vi[sel],
                                                 step=first_step + k, prec="fp32", **lw)
                    xi[sel], mi[sel], vi[sel] = a, b, c
                else:
                    a, b = O.local_sgdm_step(xi[sel], grads[i][sel], mi[sel], lr=w.local["lr"],
                                             momentum=w.local["beta1"], prec="fp32")
                    xi[sel], mi[sel] = a, b
        want[f"s1[{i}]"] = mi
        if adamw:
            want[f"s2[{i}]"] = vi
    # The global step, per tensor (the randomized sign needs each tensor's
    # bound, its index and the in-tensor element indices for Philox).
    tensors = np.unique(p)
    sel = [p == q for q in tensors]
    args = ([x0[s_] for s_ in sel], [m0[s_] for s_ in sel], [[r[s_] for s_ in sel] for r in reps])
    kw = dict(gamma=w.local["lr"], decay=[w.decay[q] for q in tensors], t=t, mode=mode,
              seed=w.philox_seed, tensor_ids=tensors, element_ids=[j[s_] for s_ in sel],
              bounds=None if B is None else [B[q] for q in tensors], **w.glob)
    o32 = O.global_step(*args, prec="fp32", **kw)
    o64 = O.global_step(*args, prec="fp64", **kw)
    want["x"], want["m"] = np.empty_like(x0), np.empty_like(m0)
    flips = outside = 0
    for a_, s_ in enumerate(sel):
        want["x"][s_], want["m"][s_] = o32["x"][a_], o32["m"][a_]
        S32, S64 = np.asarray(o32["S"][a_], np.float64), np.asarray(o64["S"][a_], np.float64)
        flip = ~((S32 == S64) | (np.isnan(S32) & np.isnan(S64)))
        if flip.any():
            u64 = np.asarray(o64["u"][a_], np.float64)
            margin = np.abs(u64[flip])
            if mode != dsm.DSM_SIGN_DET:
                U = O.randomized_sign_uniforms_at(j[s_], int(tensors[a_]), t, w.philox_seed)
                U = U[flip].astype(np.float64) * 2.0 ** -24
                thr = float(B[tensors[a_]]) * ((2 * U - 1) if mode == dsm.DSM_SIGN_RAND_FLIP else U)
                margin = np.minimum(margin, np.abs(margin - thr))
            rms_u = float(np.sqrt(np.mean(u64 * u64)))
            flips += int(flip.sum())
            outside += int(np.sum(~(margin < 1e-6 * rms_u)))
    nonbit = sum(int(np.count_nonzero(got[k].view(np.uint32) != want[k].view(np.uint32)))
                 for k in got)
    return {"elements": int(p.size), "values_compared": int(sum(v.size for v in got.values())),
            "non_bit_identical": nonbit, "flips_vs_fp64": flips,
            "flips_outside_margin": outside,
            "what": ("one untimed round of the timed path right after the timed region; x, m and "
                     "every worker's optimizer state on the sampled elements against the fp32 "
                     "oracle; sign decisions against the fp64 oracle on the same inputs")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="xl")
    ap.add_argument("--sign", choices=("det", "rand"), default="det",
                    help="global sign of the timed steps")
    ap.add_argument("--path", choices=("fused", "split"), default="fused",
                    help="fused: H-1 local steps + dsm_round_end with the lazy broadcast; "
                         "split: H local steps + dsm_global_step with broadcast")
    ap.add_argument("--extra-steps", type=int, default=20,
                    help="rounds of every path/sign combination (and launches of each variant, of "
                         "the SGD local step and of the standalone sync), timed for the breakdown")
    ap.add_argument("--flush-mb", type=int, default=0,
                    help="if > 0, also time rounds in which every call follows a write of this "
                         "many MB to a separate buffer, which evicts the arenas from the caches "
                         "(reported under breakdown_flushed; the timed steps stay unflushed)")
    ap.add_argument("--replica-layout", choices=("auto", "state-blocked", "blocked", "contiguous"),
                    default="auto",
                    help="how the per-worker buffers hold their n copies (dsm_replica_layout); "
                         "auto: state-blocked when one copy of the parameters exceeds the "
                         "256 MB last-level cache, contiguous otherwise")
    ap.add_argument("--placement", choices=("auto", "probe", "none"), default="auto",
                    help="with the state-blocked layout, place the buffers at the fastest of the "
                         "offsets of a 128 GiB larger allocation, timed at set-up (Arenas "
                         "placement_span); auto: for working sets under 120 GB")
    ap.add_argument("--no-parity", action="store_true",
                    help="skip the oracle check of one untimed round after the timed region")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="accepted for the counter runs; the plain 4 GiB device copy that "
                         "calibrates the byte counters always runs")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU exchange is a design note, not built)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2411_17866_amd import arena as A
    from paper_2411_17866_amd import dsm
    from paper_2411_17866_amd import workloads as W

    dsm.load_library()
    torch.cuda.set_device(0)
    w = W.get(args.workload)
    n, H = w.n_workers, w.local_steps
    adamw = w.base == W.BASE_ADAMW
    print(f"[bench] workload {w.name}: d={w.d} tensors={len(w.tensors)} n={n} H={H}",
          file=sys.stderr, flush=True)
    if args.replica_layout == "auto":
        # Measured on MI355X: blocking the replicas with their optimizer state
        # pins down where a kernel's streams sit in HBM, which pays once the
        # arenas stream from HBM (GPT-2 small to xl, n = 4 and 8); arenas that
        # stay in the 256 MB MALL between calls run faster contiguous (tiny
        # workload: local AdamW 20.8-21.0 us against 22.6 us).
        args.replica_layout = "state-blocked" if 4 * w.d > 256 << 20 else "contiguous"
    layout = {"state-blocked": dsm.DSM_REPLICAS_STATE_BLOCKED, "blocked": dsm.DSM_REPLICAS_BLOCKED,
              "contiguous": dsm.DSM_REPLICAS_CONTIGUOUS}[args.replica_layout]
    # Where in physical memory a working set lands sets its kernels' rate on
    # MI355X; the xl working set (125 GB) has always landed fast, smaller ones
    # often do not.  So state-blocked problems under 120 GB get the placement
    # probe, whose span (128 GiB) still fits beside them in 288 GB.
    working_set = 4 * w.d * (4 + (4 if adamw else 3) * n)
    probe = layout == dsm.DSM_REPLICAS_STATE_BLOCKED and (
        args.placement == "probe" or (args.placement == "auto" and working_set < 120e9))
    ar = A.Arenas(w.numel, n, H, w.base, decay=w.decay, randomized=True, global_adamw=True,
                  replica_layout=layout,
                  placement_span=A.PROBE_SPAN_BYTES if probe else 0)
    if ar.placement is not None:
        print("[bench] placement: offset %.1f GB, %.3f ms (slowest candidate %.3f ms) over %d "
              "candidates" % (ar.placement["offset_bytes"] / 1e9, ar.placement["best_ms"],
                              ar.placement["worst_ms"], ar.placement["candidates"]),
              file=sys.stderr, flush=True)
    gen = torch.Generator(device="cuda").manual_seed(w.seed)
    W.fill_params_(ar.x, w, gen)
    for i in range(n):
        W.fill_grads_(ar.g_rep[i], w, i, 0)
    ar.init()
    torch.cuda.synchronize()
    print("[bench] arenas resident: %.1f GB" % (torch.cuda.memory_allocated() / 1e9),
          file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    lr = w.local["lr"]
    ev = {"local": [], "local_timed": [], "local_from_x": [], "split_det": [], "split_rand": [],
          "fused_det": [],
          "fused_rand": [], "lookahead": [], "signed_slowmo": [], "global_adamw": []}
    s_count = [0]
    # After a fused round (no broadcast) every replica is stale, and the next
    # round's first local step reads x once for all workers: a different
    # kernel with fewer bytes, timed on its own.
    stale = [False]

    flush_buf = [None]

    def timed(key, fn):
        """fn between two events on the launch stream, kept under key (None:
        no events).  A pending flush (cold-cache timing) runs before."""
        if flush_buf[0] is not None:
            flush_buf[0].fill_(0.0)
        if key is None:
            fn()
            return
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        ev[key].append((e0, e1, 1))

    def one_round(t, mode, path, record=None):
        """One outer iteration.  record: None (no events); "timed" (one event
        pair around the run of ordinary local steps, so that the timed region
        holds two event records per round); "extra" (that, plus one pair
        around each other call); "flushed" (one pair around every call, each
        after a cache flush)."""
        sign = "rand" if mode else "det"
        others = record in ("extra", "flushed")
        run = []   # [start event, launches] of the open run of ordinary local steps

        def end_run():
            if run:
                e1 = torch.cuda.Event(enable_timing=True)
                e1.record(stream)
                ev["local"].append((run[0], e1, run[1]))
                if record == "timed":
                    ev["local_timed"].append((run[0], e1, run[1]))
                run.clear()

        for k in range(H):
            s_count[0] += 1
            s = s_count[0]
            if path == "fused" and k == H - 1:
                end_run()
                timed(f"fused_{sign}" if others else None,
                      lambda: dsm.dsm_round_end(ar.ctx, s, w.local, t, gamma=lr, mode=mode,
                                                seed=w.philox_seed, broadcast=False, **w.glob))
                stale[0] = True
                continue
            step = lambda: dsm.dsm_local_step(ar.ctx, -1, s, **w.local)
            if k == 0 and stale[0] and n > 1:
                timed("local_from_x" if others else None, step)
            elif record in ("timed", "extra"):
                if not run:
                    e0 = torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    run.extend([e0, 0])
                step()
                run[1] += 1
            else:
                timed("local" if record == "flushed" else None, step)
            stale[0] = False
        end_run()
        if path == "split":
            timed(f"split_{sign}" if others else None,
                  lambda: dsm.dsm_global_step(ar.ctx, t, gamma=lr, mode=mode, seed=w.philox_seed,
                                              broadcast=True, **w.glob))
            stale[0] = False

    mode_main = dsm.DSM_SIGN_DET if args.sign == "det" else dsm.DSM_SIGN_RAND_FLIP
    t = 0
    for _ in range(args.warmup):
        one_round(t, mode_main, args.path)
        t += 1
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_round(t, mode_main, args.path, "timed")
        t += 1
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print("[bench] timed steps done", file=sys.stderr, flush=True)
    # The state the timed steps produced, checked: one more round of the same
    # path, untimed, against the oracle on sampled elements.
    parity = None
    if not args.no_parity:
        parity = parity_check(w, ar, lambda: one_round(t, mode_main, args.path), t, mode_main,
                              s_count[0] + 1)
        t += 1
        print(f"[bench] parity: {parity['non_bit_identical']} of {parity['values_compared']} "
              f"values not bit-identical, {parity['flips_vs_fp64']} sign flips vs fp64",
              file=sys.stderr, flush=True)
    # Breakdown: extra rounds of every path and sign combination.
    for path in ("fused", "split"):
        for mode in (dsm.DSM_SIGN_DET, dsm.DSM_SIGN_RAND_FLIP):
            for _ in range(args.extra_steps):
                one_round(t, mode, path, "extra")
                t += 1
    torch.cuda.synchronize()

    # The same calls with cold caches: each one follows a write of flush_mb MB
    # to another buffer (outside its events), so no arena line is left in L2
    # or the MALL (Infinity Cache, 256 MB) when it starts.  This matters only
    # where the arenas fit in the caches (the tiny workload, ~80 MB).
    ev_flushed = None
    if args.flush_mb > 0:
        main_lists = {k: v for k, v in ev.items()}
        for k in ev:
            ev[k] = []
        flush_buf[0] = torch.empty(args.flush_mb * (1 << 20) // 4, dtype=torch.float32,
                                   device="cuda")
        for path in ("fused", "split"):
            for _ in range(max(1, args.extra_steps)):
                one_round(t, dsm.DSM_SIGN_DET, path, "flushed")
                t += 1
        torch.cuda.synchronize()
        flush_buf[0] = None
        ev_flushed = {k: v for k, v in ev.items()}
        ev.update(main_lists)
    ar.destroy()

    # Further contexts over the same arenas (each after the previous one is
    # destroyed, so that they never share the workspace at the same time).
    reps = max(1, args.extra_steps)
    bufs = ar.buffers()

    # The ablation variants of the global step (Section 4.1, Algorithm 7): a
    # context with H = 1, so each timed global step follows one local step.
    variants = (("lookahead", dsm.DSM_RULE_LOOKAHEAD, w.glob),
                ("signed_slowmo", dsm.DSM_RULE_SIGNED_SLOWMO, w.glob),
                ("global_adamw", dsm.DSM_RULE_GLOBAL_ADAMW,
                 dict(eta=1e-3, beta1=0.9, beta2=0.95, lam=w.glob["lam"], eps=1e-8)))
    ctx_v = dsm.dsm_init(dsm.make_problem(w.numel, n, 1, w.base, w.decay, layout), bufs)
    for key, rule, ghp in variants:
        for r in range(reps + 1):
            dsm.dsm_local_step(ctx_v, -1, r + 1, **w.local)
            timed(key if r > 0 else None,
                  lambda: dsm.dsm_global_step(ctx_v, r, gamma=lr, rule=rule, broadcast=True, **ghp))
    torch.cuda.synchronize()
    dsm.dsm_destroy(ctx_v)

    # Row a2 (local SGD + Polyak momentum, Algorithm 3) and row a6 on its own
    # (dsm_sync) at the same scale: a context with the SGD base and room for
    # reps + 1 local steps in one round.
    sgd_problem = dsm.make_problem(w.numel, n, reps + 1, dsm.DSM_BASE_SGD_MOMENTUM, w.decay,
                                   layout)
    bufs.s2_rep = None
    ctx2 = dsm.dsm_init(sgd_problem, bufs)
    ev_sgd, ev_sync = [], []
    for k in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dsm.dsm_local_step(ctx2, -1, k + 1, lr=0.1, beta1=0.9)
        e1.record(stream)
        if k > 0:
            ev_sgd.append((e0, e1, 1))
    for k in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dsm.dsm_sync(ctx2)
        e1.record(stream)
        if k > 0:
            ev_sync.append((e0, e1, 1))
    torch.cuda.synchronize()
    dsm.dsm_destroy(ctx2)

    # Practical ceiling of this device over 4 GiB buffers: torch's copy and
    # fill, and the library's pure-read and pure-write stream kernels (the
    # optimizer kernels' access shape without their arithmetic).  The read
    # kernel writes a word only for a piece whose XOR matches its pattern; a
    # piece of equal floats XORs to 0, so a non-zero pattern keeps the read
    # free of writes.
    no_match = 0x5A5A5A5A
    src = torch.zeros(1 << 30, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    words = torch.zeros(src.numel() // dsm.DSM_PIECE_ELEMS, dtype=torch.int32, device="cuda")
    sp = stream.cuda_stream

    def stream_read():
        dsm.dsm_test_stream(dsm.DSM_STREAM_READ, src.data_ptr(), src.numel(), words.data_ptr(),
                            no_match, sp)

    def stream_write():
        dsm.dsm_test_stream(dsm.DSM_STREAM_WRITE, dst.data_ptr(), dst.numel(), None, 0x40400000,
                            sp)

    dst.copy_(src)
    dst.fill_(1.0)
    stream_read()
    stream_write()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    e[0].record(stream)
    for _ in range(3):
        dst.copy_(src)
    e[1].record(stream)
    for _ in range(3):
        dst.fill_(2.0)
    e[2].record(stream)
    for _ in range(3):
        stream_read()
    e[3].record(stream)
    for _ in range(3):
        stream_write()
    e[4].record(stream)
    torch.cuda.synchronize()
    gib = 1 << 30
    copy_gbs = 3 * 8 * gib / (e[0].elapsed_time(e[1]) / 1e3) / 1e9
    fill_gbs = 3 * 4 * gib / (e[1].elapsed_time(e[2]) / 1e3) / 1e9
    sread_gbs = 3 * 4 * gib / (e[2].elapsed_time(e[3]) / 1e3) / 1e9
    swrite_gbs = 3 * 4 * gib / (e[3].elapsed_time(e[4]) / 1e3) / 1e9
    del src, dst, words

    # The same two stream kernels over the replica storage the local step
    # reads (its physical pages, which set the rate): the one block allocation
    # of the state-blocked layout, else x_rep, g_rep, s1_rep (and s2_rep).
    # Every context over the arenas is destroyed by now, so overwriting them
    # is harmless.
    rep_bufs = [ar.x_rep_flat] if ar.state_blocked else \
        [t for t in (ar.x_rep_flat, ar.g_rep, ar.s1_rep, ar.s2_rep) if t is not None]
    rep_span = 1 << 33  # elements per call, within one grid dimension
    rep_pieces = []
    for t in rep_bufs:
        flat = t.reshape(-1)
        usable = flat.numel() // dsm.DSM_PIECE_ELEMS * dsm.DSM_PIECE_ELEMS
        for o in range(0, usable, rep_span):
            rep_pieces.append((flat.data_ptr() + 4 * o, min(rep_span, usable - o)))
    rep_bytes = 4 * sum(c for _, c in rep_pieces)
    rep_read_gbs = rep_write_gbs = None
    if rep_bytes > 0:
        words = torch.empty(min(rep_span, max(c for _, c in rep_pieces)) // dsm.DSM_PIECE_ELEMS,
                            dtype=torch.int32, device="cuda")

        def rep_pass(kind, pattern):
            for ptr, c in rep_pieces:
                dsm.dsm_test_stream(kind, ptr, c, words.data_ptr(), pattern, sp)

        # The writes come first and store zeros, so the reads find no match.
        rep_pass(dsm.DSM_STREAM_WRITE, 0)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(stream)
        for _ in range(3):
            rep_pass(dsm.DSM_STREAM_WRITE, 0)
        e[1].record(stream)
        for _ in range(3):
            rep_pass(dsm.DSM_STREAM_READ, no_match)
        e[2].record(stream)
        torch.cuda.synchronize()
        rep_write_gbs = 3 * rep_bytes / (e[0].elapsed_time(e[1]) / 1e3) / 1e9
        rep_read_gbs = 3 * rep_bytes / (e[1].elapsed_time(e[2]) / 1e3) / 1e9
        del words

    def avg_ms(entries):
        """Average launch duration over (start, end, launches) event entries."""
        if not entries:
            return None
        return sum(a.elapsed_time(b) for a, b, _ in entries) / sum(c for _, _, c in entries)

    d = w.d
    khash = kernel_source_hash()
    ms_per_step = wall * 1e3 / args.steps
    updates_per_step = n * H * d + d
    value = updates_per_step / (ms_per_step / 1e3)

    def pct(vals, q):
        v = sorted(vals)
        return v[min(len(v) - 1, max(0, round(q * (len(v) - 1))))]

    def kern(entries, nbytes, updates):
        ms = avg_ms(entries)
        if ms is None:
            return None
        times = [a.elapsed_time(b) / c for a, b, c in entries]   # per launch, each entry
        gbs = nbytes / (ms / 1e3) / 1e9
        return {"ms": round(ms, 4), "GB_per_s": round(gbs, 1),
                "pct_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2),
                "param_updates_per_s": updates / (ms / 1e3), "algorithmic_bytes": nbytes,
                "launches": sum(c for _, _, c in entries), "ms_p10": round(pct(times, 0.1), 4),
                "ms_median": round(pct(times, 0.5), 4), "ms_p90": round(pct(times, 0.9), 4)}

    local_bytes = (BYTES_LOCAL_ADAMW if adamw else BYTES_LOCAL_SGDM) * n * d
    # The roofline kernel's launches inside the timed region (every other
    # local launch, when a round has no ordinary local step there).
    ms_local = avg_ms(ev["local_timed"]) or avg_ms(ev["local"])
    traffic = committed_traffic(khash, w.name, "local_adamw" if adamw else "local_sgdm")
    achieved = None if ms_local is None else local_bytes / (ms_local / 1e3) / 1e9
    shape = ("tiny parameter set" if w.name == "tiny" else f"GPT-2 {w.name}-shaped parameter set")
    local_state = 16 if adamw else 12        # x, g, s1 (, s2) read per worker
    local_written = 8 if adamw else 4        # s1 (, s2) written per worker by the round end
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "param-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{shape} ({len(w.tensors)} fp32 tensors, "
                         f"d={d}), n={n} worker replicas; one step = one outer iteration of "
                         f"Algorithm 1: H={H} local {'AdamW' if adamw else 'SGD-momentum'} steps "
                         f"on every replica + the "
                         f"{'deterministic' if args.sign == 'det' else 'randomized'}-sign global "
                         f"step ({args.path} path)"),
            "d": d, "n_workers": n, "local_steps": H, "base": "adamw" if adamw else "sgd_momentum",
            "sign": args.sign, "path": args.path, "updates_per_step": updates_per_step,
            "replica_layout": args.replica_layout,
            "placement": None if ar.placement is None else {
                "offset_GB": round(ar.placement["offset_bytes"] / 1e9, 2),
                "candidates": ar.placement["candidates"],
                "probe_ms_best": round(ar.placement["best_ms"], 3),
                "probe_ms_worst": round(ar.placement["worst_ms"], 3)},
        },
        "roofline": {
            "bound": "hbm",
            "kernel": f"k_local_{'adamw' if adamw else 'sgdm'} (dsm_local_step, all workers)",
            "achieved": None if achieved is None else round(achieved, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": None if achieved is None else round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": local_bytes,
            "avg_launch_ms": None if ms_local is None else round(ms_local, 4),
        },
        "breakdown": {
            "local_step": kern(ev["local"], local_bytes, n * d),
            "local_step_from_x": kern(ev["local_from_x"],
                                      (4 + (local_state - 4 + local_written + 4) * n) * d, n * d),
            "round_end_fused_det": kern(ev["fused_det"],
                                        (16 + (local_state + local_written) * n) * d, n * d + d),
            "round_end_fused_rand_flip": kern(ev["fused_rand"],
                                              (28 + (local_state + local_written) * n) * d,
                                              n * d + d),
            "global_det": kern(ev["split_det"], bytes_global(n, False) * d, d),
            "global_rand_flip": kern(ev["split_rand"], bytes_global(n, True) * d, d),
            "global_lookahead": kern(ev["lookahead"], bytes_global(n, False) * d, d),
            "global_signed_slowmo": kern(ev["signed_slowmo"], bytes_global(n, False) * d, d),
            "global_adamw": kern(ev["global_adamw"], (bytes_global(n, False) + 8) * d, d),
            "local_sgdm": kern(ev_sgd, BYTES_LOCAL_SGDM * n * d, n * d),
            "sync": kern(ev_sync, (4 + 4 * n) * d, n * d),
        },
        "breakdown_flushed": None if ev_flushed is None else {
            "flush_mb": args.flush_mb,
            "local_step": kern(ev_flushed["local"], local_bytes, n * d),
            "local_step_from_x": kern(ev_flushed["local_from_x"],
                                      (4 + (local_state - 4 + local_written + 4) * n) * d, n * d),
            "round_end_fused_det": kern(ev_flushed["fused_det"],
                                        (16 + (local_state + local_written) * n) * d, n * d + d),
            "global_det": kern(ev_flushed["split_det"], bytes_global(n, False) * d, d),
        },
        "device_ceiling": {"torch_copy_GB_per_s": round(copy_gbs, 1),
                           "torch_fill_GB_per_s": round(fill_gbs, 1),
                           "stream_read_GB_per_s": round(sread_gbs, 1),
                           "stream_write_GB_per_s": round(swrite_gbs, 1),
                           "replica_stream_read_GB_per_s":
                               None if rep_read_gbs is None else round(rep_read_gbs, 1),
                           "replica_stream_write_GB_per_s":
                               None if rep_write_gbs is None else round(rep_write_gbs, 1),
                           "replica_stream_GB": round(rep_bytes / 1e9, 3)},
        "kernel_source_hash": khash,
    }
    out["parity"] = parity
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, ar)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
