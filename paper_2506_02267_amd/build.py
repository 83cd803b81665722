"""Build libtav2.so (the C-ABI library) for gfx950 with hipcc, in-tree.

Usage: python -m paper_2506_02267_amd.build   (or call build()).
Every call recompiles.  Objects go to paper_2506_02267_amd/_build/, the
library to paper_2506_02267_amd/libtav2.so.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libtav2.so")
SOURCES = ["api.cpp", "batcher.cpp", "profile.cpp", "select.hip", "select_fused.hip", "gather.hip",
           "encoder_fused.hip", "encoder_fused_unmasked.hip", "encoder_small.hip",
           "encoder_f32.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libtav2)")


def compile_flags():
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Wno-unused-function", "-Wno-unused-variable",
            # keep the compiler from emitting packed-fp32 VALU instructions
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


# Per-source extra flags.  The encoders' and the fused NN search's MFMA
# results are read by VALU code (softmax, epilogues, LayerNorm, the survivor
# filter): results kept in VGPRs save one accumulator move per element (and keep
# the filter's 128 accumulators from being copied out of AGPRs all at once).  The
# d_model-64 encoder runs one wave per SIMD through chains of short dependent
# steps: the iterative ILP scheduler's order of them is 7 % faster at the paper's
# shape than the default one (the other sources gain nothing from it).  The int8
# score kernels' division and square root must round correctly (the compiler's
# default for HIP, stated explicitly).
EXTRA_FLAGS = {"encoder_fused.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
               "encoder_fused_unmasked.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
               "encoder_small.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-mllvm",
                                     "-amdgpu-sched-strategy=iterative-ilp"],
               "select.hip": ["-fhip-fp32-correctly-rounded-divide-sqrt"],
               "select_fused.hip": ["-fhip-fp32-correctly-rounded-divide-sqrt", "-mllvm",
                                    "-amdgpu-mfma-vgpr-form"]}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = ([hipcc()] + compile_flags() + EXTRA_FLAGS.get(src, [])
           + ["-c", os.path.join(CSRC, src), "-o", obj])
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines()
            if "is not a recognized feature for this target" not in ln]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n" + "\n".join(msgs))
    if msgs:
        sys.stderr.write("\n".join(msgs) + "\n")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
