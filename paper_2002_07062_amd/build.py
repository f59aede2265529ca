"""Build libbsm.so (HIP kernels for gfx950 + host planner + C ABI) in-tree.

    python -m paper_2002_07062_amd.build

Compiles every source each time it is called. hipcc cross-compiles gfx950 without a GPU.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libbsm.so")
ARCH = "gfx950"


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libbsm.so)")


def _flags() -> list[str]:
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra",
        # code object v5: loadable by every ROCm 7.x runtime, including the one torch bundles
        "-mcode-object-version=5",
        # packed fp32 VALU forms are disabled for every HIP translation unit
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        f"-I{INCLUDE}", f"-I{CSRC}",
    ]


def build(verbose: bool = False) -> str:
    hipcc = _hipcc()
    sources = ["bsm_kernels.hip", "bsm_kernels_f32.hip", "bsm_kernels_f32_shifted.hip",
               "bsm_kernels_bf16.hip", "bsm_kernels_bf16_shifted.hip", "bsm_gemm.hip",
               "bsm_noalloc.hip", "bsm_api.cpp", "bsm_plan.cpp"]
    with tempfile.TemporaryDirectory(prefix="bsm_build_") as tmp:
        def compile_one(src: str) -> str:
            obj = os.path.join(tmp, src.replace(".", "_") + ".o")
            cmd = [hipcc, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj] + _flags()
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
            if verbose and r.stderr.strip():
                print(r.stderr, file=sys.stderr)
            return obj

        with ThreadPoolExecutor(max_workers=len(sources)) as ex:
            objs = list(ex.map(compile_one, sources))
        out_tmp = LIB + ".tmp"
        cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out_tmp] + objs + [
            "-Wl,-soname,libbsm.so"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"linking libbsm.so failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
        os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
