"""Python binding of the C ABI in include/dsm.h (argument marshalling only).

Every function has the name of the C entry point it calls and does no
arithmetic of the method: each step of the path runs in the HIP kernels of
libdsm.so.  Loading fails loudly when the library has not been built; there
is no fallback.
"""
import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBPATH = os.path.join(_PKG, "lib", "libdsm.so")

DSM_OK = 0
DSM_ERR_INVALID_ARG = 1
DSM_ERR_STATE = 2
DSM_ERR_HIP = 3
DSM_ERR_UNSUPPORTED = 4
STATUS_NAMES = {0: "DSM_OK", 1: "DSM_ERR_INVALID_ARG", 2: "DSM_ERR_STATE", 3: "DSM_ERR_HIP",
                4: "DSM_ERR_UNSUPPORTED"}

DSM_BASE_ADAMW = 0
DSM_BASE_SGD_MOMENTUM = 1

DSM_SIGN_DET = 0
DSM_SIGN_RAND_FLIP = 1
DSM_SIGN_RAND_ZERO = 2

DSM_RULE_SIGN_MOMENTUM = 0
DSM_RULE_LOOKAHEAD = 1
DSM_RULE_SIGNED_SLOWMO = 2
DSM_RULE_GLOBAL_ADAMW = 3

DSM_REPLICAS_CONTIGUOUS = 0
DSM_REPLICAS_BLOCKED = 1
DSM_REPLICAS_STATE_BLOCKED = 2
DSM_REPLICA_BLOCK_ELEMS = 16384
DSM_STATE_BLOCK_ELEMS = 4096
DSM_PIECE_ELEMS = 1024
DSM_STREAM_READ, DSM_STREAM_WRITE = 0, 1

EXPORTED = ("dsm_layout", "dsm_init", "dsm_init_static", "dsm_local_step", "dsm_global_step",
            "dsm_round_end", "dsm_sync",
            "dsm_read_bounds", "dsm_test_philox", "dsm_test_stream", "dsm_destroy",
            "dsm_last_error")


class DsmError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class dsm_problem(ctypes.Structure):
    _fields_ = [("n_workers", ctypes.c_int32), ("local_steps", ctypes.c_int32),
                ("n_tensors", ctypes.c_int32), ("base", ctypes.c_int32),
                ("numel", ctypes.POINTER(ctypes.c_int64)),
                ("decay", ctypes.POINTER(ctypes.c_uint8)),
                ("replica_layout", ctypes.c_int32)]


class dsm_buffers(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("m", ctypes.c_void_p), ("x_rep", ctypes.c_void_p),
                ("g_rep", ctypes.c_void_p), ("s1_rep", ctypes.c_void_p),
                ("s2_rep", ctypes.c_void_p), ("u_scratch", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_int64),
                ("stream", ctypes.c_void_p), ("v", ctypes.c_void_p)]


class dsm_local_hparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


class dsm_global_hparams(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_float), ("eta", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("lambda_", ctypes.c_float), ("mode", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("rule", ctypes.c_int32), ("eps", ctypes.c_float)]


_lib = None


def load_library(path=LIBPATH):
    """Loads libdsm.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} not found: build the HIP library first "
                           "(python -m paper_2411_17866_amd.build)")
    lib = ctypes.CDLL(path)
    c_int64_p = ctypes.POINTER(ctypes.c_int64)
    lib.dsm_layout.argtypes = [ctypes.POINTER(dsm_problem), c_int64_p, c_int64_p, c_int64_p]
    lib.dsm_init.argtypes = [ctypes.POINTER(dsm_problem), ctypes.POINTER(dsm_buffers),
                             ctypes.POINTER(ctypes.c_void_p)]
    lib.dsm_init_static.argtypes = [ctypes.POINTER(dsm_problem), ctypes.POINTER(dsm_buffers),
                                    ctypes.POINTER(ctypes.c_void_p)]
    lib.dsm_local_step.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                   ctypes.POINTER(dsm_local_hparams)]
    lib.dsm_global_step.argtypes = [ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.POINTER(dsm_global_hparams), ctypes.c_int32]
    lib.dsm_round_end.argtypes = [ctypes.c_void_p, ctypes.c_int64,
                                  ctypes.POINTER(dsm_local_hparams), ctypes.c_int64,
                                  ctypes.POINTER(dsm_global_hparams), ctypes.c_int32]
    lib.dsm_sync.argtypes = [ctypes.c_void_p]
    lib.dsm_read_bounds.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_float),
                                    ctypes.c_int32]
    lib.dsm_test_philox.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                    ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p]
    lib.dsm_test_stream.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p]
    lib.dsm_destroy.argtypes = [ctypes.c_void_p]
    lib.dsm_last_error.argtypes = [ctypes.c_void_p]
    lib.dsm_last_error.restype = ctypes.c_char_p
    for name in EXPORTED:
        if name != "dsm_last_error":
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def dsm_last_error(ctx=None):
    return load_library().dsm_last_error(ctx).decode()


def _check(status, ctx=None):
    if status != DSM_OK:
        raise DsmError(status, dsm_last_error(ctx))


def make_problem(numel, n_workers, local_steps, base, decay=None,
                 replica_layout=DSM_REPLICAS_CONTIGUOUS):
    """A dsm_problem plus the host arrays it points to (kept alive with it)."""
    numel = np.ascontiguousarray(np.asarray(numel, dtype=np.int64))
    keep = [numel]
    prob = dsm_problem(n_workers, local_steps, len(numel), base,
                       numel.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), None,
                       replica_layout)
    if decay is not None:
        dec = np.ascontiguousarray(np.asarray(decay, dtype=np.uint8))
        keep.append(dec)
        prob.decay = dec.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))
    prob._keep = keep
    return prob


def dsm_layout(problem):
    """Returns (arena_elems, tensor_offsets, workspace_bytes)."""
    lib = load_library()
    arena = ctypes.c_int64()
    ws = ctypes.c_int64()
    offs = np.zeros(max(problem.n_tensors, 1), dtype=np.int64)
    _check(lib.dsm_layout(ctypes.byref(problem), ctypes.byref(arena),
                          offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), ctypes.byref(ws)))
    return arena.value, offs[:problem.n_tensors].copy(), ws.value


def dsm_init(problem, buffers):
    """Returns the context handle (an opaque pointer value)."""
    lib = load_library()
    ctx = ctypes.c_void_p()
    _check(lib.dsm_init(ctypes.byref(problem), ctypes.byref(buffers), ctypes.byref(ctx)))
    return ctx.value


def dsm_init_static(problem, buffers):
    """dsm_init with the workspace and u staging in the library's static
    scratch (buffers.workspace and u_scratch are ignored)."""
    lib = load_library()
    ctx = ctypes.c_void_p()
    _check(lib.dsm_init_static(ctypes.byref(problem), ctypes.byref(buffers), ctypes.byref(ctx)))
    return ctx.value


def dsm_local_step(ctx, worker, step, lr, beta1, beta2=0.0, eps=0.0, weight_decay=0.0):
    hp = dsm_local_hparams(lr, beta1, beta2, eps, weight_decay)
    _check(load_library().dsm_local_step(ctx, worker, step, ctypes.byref(hp)), ctx)


def dsm_global_step(ctx, t, gamma, eta, beta1, beta2, lam, mode=DSM_SIGN_DET, seed=0,
                    broadcast=True, rule=DSM_RULE_SIGN_MOMENTUM, eps=1e-8):
    hp = dsm_global_hparams(gamma, eta, beta1, beta2, lam, mode, seed, rule, eps)
    _check(load_library().dsm_global_step(ctx, t, ctypes.byref(hp), 1 if broadcast else 0), ctx)


def dsm_round_end(ctx, step, local, t, gamma, eta, beta1, beta2, lam, mode=DSM_SIGN_DET, seed=0,
                  broadcast=True, rule=DSM_RULE_SIGN_MOMENTUM, eps=1e-8):
    """local: dict of dsm_local_hparams fields (lr, beta1, beta2, eps, weight_decay)."""
    lhp = dsm_local_hparams(local["lr"], local["beta1"], local.get("beta2", 0.0),
                            local.get("eps", 0.0), local.get("weight_decay", 0.0))
    ghp = dsm_global_hparams(gamma, eta, beta1, beta2, lam, mode, seed, rule, eps)
    _check(load_library().dsm_round_end(ctx, step, ctypes.byref(lhp), t, ctypes.byref(ghp),
                                        1 if broadcast else 0), ctx)


def dsm_sync(ctx):
    _check(load_library().dsm_sync(ctx), ctx)


def dsm_read_bounds(ctx, n_tensors):
    """The bounds of the last randomized global step; n_tensors is the size of
    the array handed to the library (the call fails if the problem has more)."""
    out = np.zeros(max(n_tensors, 1), dtype=np.float32)
    _check(load_library().dsm_read_bounds(ctx, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                          out.size), ctx)
    return out[:n_tensors]


def dsm_test_philox(seed, tensor, t, q0, count, dev_out_ptr, stream_ptr=None):
    _check(load_library().dsm_test_philox(seed, tensor, t, q0, count, dev_out_ptr, stream_ptr))


def dsm_test_stream(kind, dev_buf_ptr, n_elems, dev_words_ptr=None, pattern=0, stream_ptr=None):
    _check(load_library().dsm_test_stream(kind, dev_buf_ptr, n_elems, dev_words_ptr, pattern,
                                          stream_ptr))


def dsm_destroy(ctx):
    _check(load_library().dsm_destroy(ctx))
