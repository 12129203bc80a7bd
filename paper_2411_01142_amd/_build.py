"""Build libneoattn.so in-tree with hipcc for gfx950."""
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
LIB = os.path.join(PKG, "libneoattn.so")
BUILD_DIR = os.path.join(PKG, "_build")

SOURCES = ["api.hip", "plan_combine.hip", "decode_mfma.hip", "decode_valu.hip", "kv_ops.hip"]
# Host-only C++ (the CPU attention, the scheduler, the error text), built with
# the host compiler; the CPU attention's ISA-specific functions carry target
# attributes and are picked at run time.
HOST_SOURCES = ["cpu_attention.cpp", "scheduler.cpp", "neo_error.cpp"]
HOST_FLAGS = ["-O3", "-fPIC", "-std=c++17", "-Wall", "-pthread", "-fno-math-errno",
              "-I" + INCLUDE, "-I" + CSRC]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall",
    "-I" + INCLUDE, "-I" + CSRC,
    # No packed fp32 arithmetic in device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
# Per-source additions. The decode kernel's first four arguments (five dwords:
# lengths pointer, batch, kv heads, table stride) arrive preloaded in SGPRs,
# so each wave's first length read goes out without waiting for a
# kernel-argument load.
HIPCC_SOURCE_FLAGS = {
    "decode_mfma.hip": ["-mllvm", "-amdgpu-kernarg-preload-count=4"],
}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; libneoattn needs ROCm's hipcc to build")


def cxx() -> str:
    for cand in (os.environ.get("CXX"), shutil.which("g++"), shutil.which("c++")):
        if cand:
            return cand
    raise RuntimeError("no host C++ compiler (g++) found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    if src in HOST_SOURCES:
        cmd = [cxx(), *HOST_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    else:
        cmd = [hipcc(), *HIPCC_FLAGS, *HIPCC_SOURCE_FLAGS.get(src, []), "-c",
               os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stdout}\n{res.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link libneoattn.so (always rebuilds)."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = SOURCES + HOST_SOURCES
    with cf.ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-pthread", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
