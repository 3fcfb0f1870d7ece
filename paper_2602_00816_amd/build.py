"""Build the HIP library libfdhvp.so for gfx950, in-tree.

Every source under csrc/ is compiled with hipcc (packed-fp32 code generation
disabled) into an object, in parallel, and linked into one shared library next
to this file.  Usage: ``python -m paper_2602_00816_amd.build [--incremental]``
or ``build()``.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libfdhvp.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(os.path.dirname(HERE), "include")]

SOURCES = ["gemm.hip", "attn.hip", "rng.hip", "vec.hip", "lm.hip", "engine.hip", "capi.hip"]
# The fused attention kernels keep their MFMA accumulators in VGPRs: with the
# default AGPR form the allocator moves the output accumulators through VGPRs
# around every score product.
EXTRA = {"attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _headers_mtime() -> float:
    inc = os.path.join(os.path.dirname(HERE), "include")
    paths = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    paths += [os.path.join(inc, f) for f in os.listdir(inc) if f.endswith(".h")]
    return max(os.path.getmtime(p) for p in paths)


def _compile(src: str, incremental: bool = False, hdr: float = 0.0) -> str:
    obj = os.path.join(OUT, os.path.splitext(src)[0] + ".o")
    if incremental and os.path.exists(obj):
        t = os.path.getmtime(obj)
        if t >= os.path.getmtime(os.path.join(CSRC, src)) and t >= hdr:
            return obj
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-6000:]}")
    return obj


def build(verbose: bool = False, incremental: bool = False) -> str:
    """Compile every source (or, with incremental, only those whose object is
    older than the source or any header) and link the library."""
    os.makedirs(OUT, exist_ok=True)
    workers = min(len(SOURCES), max(1, (os.cpu_count() or 2)))
    hdr = _headers_mtime()
    with cf.ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(lambda f: _compile(f, incremental, hdr), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-6000:]}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True, incremental="--incremental" in sys.argv)
    sys.exit(0)
