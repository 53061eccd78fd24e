"""Builds libnmd.so (the C ABI of include/nmd.h) in-tree for gfx950 with hipcc.

    python -m paper_2608_21607_amd.build [-v]

Every source is compiled to an object under _build/ (in parallel), then linked into
paper_2608_21607_amd/libnmd.so next to this file.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnmd.so")
SOURCES = ["host.cpp", "ingest.cpp", "dense.hip", "dense_bf16.hip", "dense_large.hip", "dense_bf16_large.hip",
           "objective.hip", "sparse.hip", "solve.hip", "chol.hip", "layout.hip", "noalloc.hip"]
ARCH = "gfx950"

# Packed-fp32 instructions are kept out of the generated code on purpose.
HIPFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result",
    "-I", os.path.join(ROOT, "include"),
]


# Per-source additions.  The dense kernel for r_p <= 256 keeps its MFMA accumulators in ordinary
# VGPRs: with accumulation registers the compiler copies the output tiles between the two
# register files on every panel block at small ranks (measured: r = 16 at 53% of the fp32 MFMA
# peak instead of 72%).  The r_p >= 320 instantiations (dense_large.hip) keep the default: at
# one wave per SIMD the output tiles sit in accumulation registers and leave the VGPRs to the
# operands (r = 512: 3-4% faster).  The split-bf16 kernels follow the fp32 ones: dense_bf16.hip
# (r_p <= 256) with the VGPR form, dense_bf16_large.hip (r_p = 512) with the default.
EXTRA_FLAGS = {"dense.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
               "dense_bf16.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str, obj: str, verbose: bool) -> None:
    cmd = [hipcc(), *HIPFLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    if verbose and res.stderr.strip():
        print(res.stderr, flush=True)


def build(verbose: bool = False) -> str:
    """Compiles every source and links libnmd.so; returns its path."""
    out_dir = os.path.join(ROOT, "_build")
    os.makedirs(out_dir, exist_ok=True)
    objs = [os.path.join(out_dir, s.rsplit(".", 1)[0] + ".o") for s in SOURCES]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        list(ex.map(lambda p: _compile(p[0], p[1], verbose), zip(SOURCES, objs)))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
