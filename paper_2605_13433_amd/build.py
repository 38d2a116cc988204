"""Builds libhstu_jagged.so (HIP kernels + C ABI) for gfx950, in-tree.

Every translation unit is compiled by hipcc with packed fp32 vector ops
disabled (-Xclang -target-feature -Xclang -packed-fp32-ops) and with
hardware float atomics on device memory (-munsafe-fp-atomics), then linked
into one shared library next to this file.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libhstu_jagged.so")
ARCH = "gfx950"
SOURCES = ["api.cpp", "sched.hip", "attn_bf16.hip", "attn_f32.hip", "norm.hip",
           "layer.cpp", "layer_kernels.hip", "noalloc.hip", "embedding.hip", "rab.hip",
           "gemm.hip"]
HEADERS = ["device.h", "internal.h", "sched_impl.h"]

CFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-munsafe-fp-atomics", "-Wall", "-Wno-unused-function",
          "-Wno-unused-variable"]


# Per-file flags.  The attention kernels' only uniform-address atomic is a
# work-group's one-lane pop of its next item; the compiler's atomic
# optimizer would wrap it in a wave-wide reduction whose broadcast of the
# returned value waits for the atomic at once (and with it for every load
# and atomic in flight), instead of where the value is first used, a step
# later.
FILE_FLAGS = {"attn_bf16.hip": ["-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]}

# The layer shell's GEMMs run on hipBLASLt.
LDFLAGS = ["-L/opt/rocm/lib", "-lhipblaslt"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [_hipcc(), *CFLAGS, *FILE_FLAGS.get(src, []), "-x", "hip", "-c",
           os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compiles every source (always) and links LIB; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    workers = min(len(SOURCES), max(1, (os.cpu_count() or 4)), 8)
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs,
           *LDFLAGS, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
