"""Build libbd.so (the gfx950 HIP kernels and their C ABI) in-tree with hipcc.

Usage: ``python -m paper_2606_00144_amd.build`` or ``build_library()``.
Every source is compiled to its own object in parallel, then linked.

``python -m paper_2606_00144_amd.build --host-sanitize`` builds a second copy,
``_build_san/libbd.so``, whose host code (argument checks, planning, workspace
sizes) carries AddressSanitizer and UndefinedBehaviorSanitizer; the GPU code is
built as usual.  It is for checking the C ABI on the CPU: load it with
``BD_LIBRARY=<path>`` and the sanitizer runtime preloaded (``LD_PRELOAD`` of
clang's ``libclang_rt.asan-x86_64.so``).
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libbd.so")
SAN_BUILD = os.path.join(PKG, "_build_san")
SAN_LIB = os.path.join(SAN_BUILD, "libbd.so")

SOURCES = ["attn.hip", "attn_bwd.hip", "select.hip", "accept.hip", "update.hip", "ce.hip", "bd_api.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    "-x", "hip", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from forming packed-fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs: the kernels fit in 256 of them, and accumulators in
    # AGPRs make the compiler copy them to VGPRs around every conditional rescale
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
# host pass only: each sanitizer flag is preceded by -Xarch_host, so no GPU code is instrumented
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer"]


def _compile(src: str, build_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build_library(verbose: bool = False, host_sanitize: bool = False) -> str:
    build_dir, lib = (SAN_BUILD, SAN_LIB) if host_sanitize else (BUILD, LIB)
    extra = HOST_SANITIZE if host_sanitize else []
    os.makedirs(build_dir, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, extra), SOURCES))
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build_library(verbose=True, host_sanitize="--host-sanitize" in sys.argv[1:])
    sys.exit(0)
