"""Builds libzf.so (the HIP library behind include/zf.h) in-tree for gfx950.

    python paper_2505_12242_amd/build.py

(run as a script: importing the package loads the library it is about to
rebuild).  Each source is compiled to an object file in parallel, then
linked.

Flags: -ffp-contract=off and correctly rounded fp32 division / square root
keep every arithmetic line of the kernels a single IEEE operation; packed
fp32 instructions are disabled.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libzf.so")
ARCH = "gfx950"

SOURCES = ["zf_api.hip", "zf_kernels.hip", "zf_kernels_cm.hip", "zf_kernels_zen.hip",
           "zf_kernels_offload.hip", "zf_kernels_rv.hip", "zf_kernels_stream.hip", "zf_host.cpp"]

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall", "-pthread",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found (ROCm is required to build libzf)")
    return path


OBJ_DIR = os.path.join(ROOT, "_build")


def _run(cmd, verbose, what):
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        sys.stderr.write(proc.stdout + proc.stderr)
        raise RuntimeError(f"hipcc failed on {what} (exit code {proc.returncode})")
    noise = [ln for ln in (proc.stdout + proc.stderr).splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln]
    if verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    compile_flags = [f for f in FLAGS if f != "-shared"]
    objs = [os.path.join(OBJ_DIR, os.path.splitext(src)[0] + ".o") for src in SOURCES]

    def compile_one(i):
        _run([hipcc(), *compile_flags, "-I", INCLUDE, "-I", CSRC, "-c",
              os.path.join(CSRC, SOURCES[i]), "-o", objs[i]], verbose, SOURCES[i])

    jobs = max(1, min(len(SOURCES), os.cpu_count() or 1))
    with ThreadPoolExecutor(jobs) as ex:
        list(ex.map(compile_one, range(len(SOURCES))))
    tmp = LIB + ".tmp"
    _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-pthread", "-o", tmp, *objs],
         verbose, "the link of libzf.so")
    os.replace(tmp, LIB)
    build_abi_smoke(verbose)
    return LIB


ABI_SMOKE_SRC = os.path.join(ROOT, "tests", "abi", "abi_smoke.cpp")
ABI_SMOKE_BIN = os.path.join(ROOT, "tests", "abi", "abi_smoke")


def build_abi_smoke(verbose: bool = False) -> str:
    """The C++ consumer of the C ABI used by the native GPU test (links
    libzf.so from the package directory through its rpath)."""
    if not os.path.exists(ABI_SMOKE_SRC):
        return ""
    tmp = ABI_SMOKE_BIN + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O2", "-std=c++17", "-Wall", "-I", INCLUDE,
           ABI_SMOKE_SRC, "-L", PKG, "-lzf", "-Wl,-rpath,$ORIGIN/../../paper_2505_12242_amd",
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        sys.stderr.write(proc.stdout + proc.stderr)
        raise RuntimeError(f"hipcc failed on the ABI smoke program (exit {proc.returncode})")
    os.replace(tmp, ABI_SMOKE_BIN)
    return ABI_SMOKE_BIN


if __name__ == "__main__":
    print(build(verbose=True))
