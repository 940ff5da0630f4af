"""Builds libdsm.so (the C-ABI library of include/dsm.h) for gfx950 with hipcc.

    python -m paper_2411_17866_amd.build

Output: paper_2411_17866_amd/lib/libdsm.so.  Intermediate objects go to
_build/ at the repository root.  Every call compiles from source.
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "lib")
OBJDIR = os.path.join(ROOT, "_build")
LIBPATH = os.path.join(LIBDIR, "libdsm.so")

ARCH = "gfx950"
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

# Numerics: one IEEE fp32 rounding per written operation (no FMA contraction),
# correctly rounded division and square root, denormals kept.  Packed fp32
# instructions are disabled.
COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wextra",
    "-Wno-unused-parameter",
    "-ffp-contract=off",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
DEVICE_FLAGS = [
    f"--offload-arch={ARCH}",
    "-fno-gpu-flush-denormals-to-zero",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; the library needs ROCm's hipcc to build")
    return exe


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose=False, out=LIBPATH, defines=()):
    """Compiles the kernels and the host runtime and links libdsm.so.

    defines: extra -D settings of the build-time tuning knobs (DSM_BLOCK_THREADS,
    DSM_UNROLL, DSM_ITERS, DSM_NT, DSM_CHUNK_ELEMS, and the XCD maps of each
    replica layout DSM_MAPS_CONTIGUOUS, DSM_MAPS_BLOCKED, DSM_MAPS_STATE_BLOCKED
    as "local, round_end, from_x, global, copy"); the defaults are the tuned
    values.
    """
    os.makedirs(os.path.dirname(out), exist_ok=True)
    objdir = os.path.join(OBJDIR, "_".join(d.replace("=", "") for d in defines) or "default")
    os.makedirs(objdir, exist_ok=True)
    dflags = [f"-D{d}" for d in defines]
    cc = hipcc()
    k_obj = os.path.join(objdir, "dsm_kernels.o")
    r_obj = os.path.join(objdir, "dsm_runtime.o")
    _run([cc, "-x", "hip", *COMMON_FLAGS, *DEVICE_FLAGS, *dflags, "-c",
          os.path.join(CSRC, "dsm_kernels.hip"), "-o", k_obj], verbose)
    _run([cc, "-x", "c++", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", *COMMON_FLAGS,
          *dflags, "-c", os.path.join(CSRC, "dsm_runtime.cpp"), "-o", r_obj], verbose)
    tmp = out + ".tmp"
    _run([cc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, k_obj, r_obj,
          "-Wl,--no-undefined", "-Wl,-soname,libdsm.so"], verbose)
    os.replace(tmp, out)
    return out


def kernel_isa(path=None):
    """Writes the gfx950 assembly of the kernels, compiled with the library's flags, for review."""
    out = path or os.path.join(OBJDIR, "dsm_kernels.s")
    _run([hipcc(), "-x", "hip", *COMMON_FLAGS, *DEVICE_FLAGS, "--offload-device-only", "-S",
          os.path.join(CSRC, "dsm_kernels.hip"), "-o", out], False)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
