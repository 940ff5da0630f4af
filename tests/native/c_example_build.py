"""Builds tests/native/c_abi_example.c: the C ABI used from plain C (gcc, no
Python or torch on the path).  The binary goes to tests/native/bin/ and finds
libdsm.so through its run path."""
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SRC = os.path.join(HERE, "c_abi_example.c")
EXE = os.path.join(HERE, "bin", "c_abi_example")


def build():
    """Compiles the example; returns its path (None without a C compiler)."""
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        return None
    os.makedirs(os.path.dirname(EXE), exist_ok=True)
    libdir = os.path.join(ROOT, "paper_2411_17866_amd", "lib")
    cmd = [cc, "-std=c99", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}", SRC,
           f"-L{libdir}", "-ldsm", f"-L{ROCM}/lib", "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../../paper_2411_17866_amd/lib", f"-Wl,-rpath,{ROCM}/lib",
           "-o", EXE]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building the C ABI example failed:\n{r.stderr}")
    return EXE


if __name__ == "__main__":
    print(build())
