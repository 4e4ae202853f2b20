"""Compile the HIP sources under csrc/ into paper_2609_39056_amd/lib/libsq.so
for gfx950 (cross-compiles without a GPU)."""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libsq.so")
OBJDIR = os.path.join(ROOT, "_build", "obj")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# -ffp-contract=off: the quantizer's fp32 chain must not be fused into FMAs
#   (the kernels request FMAs explicitly where they want them);
# correctly rounded fp32 divide (the scale chain uses c / q_max and 1 / Delta);
# IEEE denormals; no packed-fp32 instruction selection.
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep MFMA accumulators in arch VGPRs (the dequantization reads them with
    # plain VALU ops) and never spill private arrays into LDS
    "-mllvm", "-amdgpu-mfma-vgpr-form", "-mllvm", "-disable-promote-alloca-to-lds",
    "-Wall", "-Wno-unused-function",
    f"-I{INCLUDE}", f"-I{CSRC}",
]

SOURCES = ["sq_api.cpp", "quant_act.hip", "pack_weights.hip", "gemm_w4.hip", "gemm_skinny.hip", "unfused.hip",
           "mfma_probe.hip", "calib.hip", "noalloc.hip", "gelu.hip"]


_REMARK = re.compile(r"remark: Function Name: (\S+)|remark:\s+(ScratchSize \[bytes/lane\]|VGPRs Spill): (\d+)")


def _check_resources(src: str, stderr: str) -> None:
    """Every kernel must keep its working set in registers and LDS: any
    scratch (private memory) use or vector-register spill fails the build.
    (Scalar registers spill into vector-register lanes, not memory.)"""
    kernel, bad = None, []
    for m in _REMARK.finditer(stderr):
        if m.group(1):
            kernel = m.group(1)
        elif int(m.group(3)) != 0:
            bad.append(f"{kernel}: {m.group(2)} = {m.group(3)}")
    if bad:
        raise RuntimeError(f"{src}: kernels use scratch memory or spill registers:\n  " + "\n  ".join(bad))


def _compile(src: str) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-Rpass-analysis=kernel-resource-usage", "-x", "hip", "-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if src.endswith(".hip"):
        _check_resources(src, r.stderr)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source (always) and link libsq.so; returns its path."""
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
