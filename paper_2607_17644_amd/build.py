"""Compile the gfx950 HIP sources into the in-tree shared library liblaga.so.

Usage: python paper_2607_17644_amd/build.py   (standalone: it does not import the package,
whose import needs the built library)
Every call recompiles (sources are few and hipcc is fast); objects go to
paper_2607_17644_amd/_build/, the library to paper_2607_17644_amd/liblaga.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "liblaga.so")
ARCH = "gfx950"

SOURCES = ["api.hip", "gemm.hip", "attn_fwd.hip", "attn_bwd.hip", "attn_bwd_kv.hip", "attn_bwd_dq.hip", "prologue.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-fvisibility=hidden",
    # packed fp32 ops are disabled: hand-written float code must not become v_pk_*_f32
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


# Per-file code-generation choices (measured: with MFMA results kept in VGPRs the
# softmax / dZ arithmetic on the accumulators needs no AGPR<->VGPR copies).
EXTRA = {
    "attn_fwd.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "attn_bwd_dq.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "attn_bwd_kv.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    demo = build_c_consumer()
    if verbose:
        print(f"built {demo}")
    return LIB


# A plain C program that uses only include/laga.h and the HIP runtime's C API (the GPU
# tests run it to show that the boundary needs no PyTorch and no C++).
C_DEMO_SRC = os.path.join(ROOT, "tests", "c_consumer", "laga_c_demo.c")
C_DEMO = os.path.join(BUILD, "laga_c_demo")


def build_c_consumer() -> str:
    os.makedirs(BUILD, exist_ok=True)
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(HIPCC)))
    cmd = [os.environ.get("CC", "gcc"), "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", os.path.join(rocm, "include"),
           C_DEMO_SRC, "-o", C_DEMO, "-L", PKG, "-llaga", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/..", "-Wl,-rpath," + os.path.join(rocm, "lib"), "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"C consumer build failed:\n{' '.join(cmd)}\n{r.stderr}")
    return C_DEMO


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
