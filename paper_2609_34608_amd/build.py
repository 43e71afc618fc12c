"""Build libwam.so for gfx950 in-tree with hipcc.

    python -m paper_2609_34608_amd.build

Each HIP translation unit under csrc/ is compiled separately (in parallel)
and linked into paper_2609_34608_amd/lib/libwam.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libwam.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ROCM_LIB = "/opt/rocm/lib"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    # packed fp32 instructions are kept out of generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators stay in architectural VGPRs: with the default
    # heuristic, unrolled loops shuffle accumulators between AGPRs and VGPRs
    # with several copy instructions per MFMA
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}",
]

SOURCES = ["k_small.hip", "k_gemm.hip", "k_attention.hip", "k_probe.hip", "wam_api.hip"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    # roctx ranges (phase annotations for marker traces) come from the ROCm
    # profiler SDK's small roctx library
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs, f"-L{ROCM_LIB}",
           "-lrocprofiler-sdk-roctx", f"-Wl,-rpath,{ROCM_LIB}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


HOSTSAN = os.path.join(BUILD, "hostsan")
HOST_CHECK_SRC = os.path.join(ROOT, "tests", "host", "abi_host_check.cpp")
CLANGXX = "/opt/rocm/llvm/bin/clang++"


def build_host_check() -> str:
    """The host ABI check program (tests/host/abi_host_check.cpp) linked
    against the library objects with AddressSanitizer and
    UndefinedBehaviorSanitizer on their host code; the device code is built
    as usual.  Objects are rebuilt only when a source changed."""
    os.makedirs(HOSTSAN, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]

    def one(src: str) -> str:
        path = os.path.join(CSRC, src)
        obj = os.path.join(HOSTSAN, os.path.splitext(src)[0] + ".o")
        deps = [path] + [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")] + \
               [os.path.join(INCLUDE, "wam.h")]
        if os.path.exists(obj) and os.path.getmtime(obj) >= max(os.path.getmtime(d) for d in deps):
            return obj
        cmd = [HIPCC, *COMMON, *san, "-c", path, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (host sanitizers) failed for {src}:\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(one, SOURCES))
    exe = os.path.join(HOSTSAN, "abi_host_check")
    drv = os.path.join(HOSTSAN, "abi_host_check.o")
    sanflags = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-g"]
    for cmd in ([CLANGXX, "-O1", *sanflags, f"-I{INCLUDE}", "-c", HOST_CHECK_SRC, "-o", drv],
                [CLANGXX, *sanflags, drv, *objs, f"-L{ROCM_LIB}", "-lamdhip64", "-lrocprofiler-sdk-roctx",
                 f"-Wl,-rpath,{ROCM_LIB}", "-o", exe]):
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"host check build failed:\n{' '.join(cmd)}\n{r.stderr}")
    return exe


def clean():
    shutil.rmtree(BUILD, ignore_errors=True)


if __name__ == "__main__":
    build()
    sys.exit(0)
