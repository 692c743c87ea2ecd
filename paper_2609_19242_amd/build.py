"""Build the HIP library ``libbdlm_attn.so`` for gfx950 with hipcc.

Every source under ``csrc/`` is compiled to an object in ``_build/`` (in
parallel) and linked into ``libbdlm_attn.so`` next to this file.  Packed-fp32
instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libbdlm_attn.so")
BUILD_DIR = os.path.join(HERE, "_build")
SOURCES = ["api.cpp", "fwd_bf16.hip", "fwd_f32.hip", "merge.hip", "bwd_pre.hip", "bwd_bf16.hip", "bwd_dkdv.hip",
           "bwd_dq.hip", "bwd_f32.hip"]
ARCH = os.environ.get("BDLM_OFFLOAD_ARCH", "gfx950")
# Per-source code-generation options.  The dK/dV kernel runs one wave per SIMD,
# so its speed is its own instruction stream: the iterative ILP scheduler keeps
# more LDS reads in flight, and VGPR-form MFMAs stop the register allocator from
# sharing AGPRs between the per-step S/dP tiles and the dK/dV accumulators
# (about 190 -> 70 register-file copies per step).  Measured at L=32768:
# 44.4 -> 42.9 -> 38.9 ms; both are slower for the two-waves-per-SIMD kernels.
EXTRA_FLAGS = {"bwd_bf16.hip": ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp", "-mllvm", "-amdgpu-mfma-vgpr-form"],
               # score and dP accumulators in VGPRs (the softmax reads them); the
               # dK/dV accumulators are AGPR operands of inline-assembly MFMAs
               "bwd_dkdv.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def flags() -> list:
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
        "-Wno-unused-command-line-argument",
    ]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *flags(), *EXTRA_FLAGS.get(src, []), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
