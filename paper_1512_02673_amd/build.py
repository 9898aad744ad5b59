"""Builds the HIP library (libcoded_mi355x.so) in-tree for gfx950 with hipcc.

Every call recompiles every source; objects go to _build/ next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB_NAME = "libcoded_mi355x.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
ARCH = "gfx950"

SOURCES = ["api.cpp", "survivors.cpp", "shuffle.cpp", "encode.hip", "worker.hip", "worker_f32_mfma.hip", "worker_bf16.hip", "fused_bf16.hip",
           "decode.hip", "onepass.hip", "transpose.hip", "runtime.hip", "shuffle.hip", "scratch.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result", f"-I{os.path.join(ROOT, 'include')}"]
# Device code: gfx950 only; packed-fp32 instructions disabled.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# Kernels that accumulate on the matrix cores in loops: keep the accumulators
# in vector registers (otherwise the compiler copies them to and from the
# accumulation registers around loop iterations, vector instructions that do
# not overlap with the fp64 matrix work; the fp32 products at s = 16..64
# measured 5% faster, the others unchanged).
MFMA_VGPR_FORM = {"worker_f32_mfma.hip", "decode.hip", "worker_bf16.hip"}


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, src + ".o")
    path = os.path.join(CSRC, src)
    if src.endswith(".hip"):
        extra = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"] if src in MFMA_VGPR_FORM else []
        cmd = [hipcc(), "-x", "hip", *DEVICE, *extra, *COMMON, "-c", path, "-o", obj]
    else:
        cmd = [hipcc(), *COMMON, "-D__HIP_PLATFORM_AMD__", "-c", path, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{res.stdout}\n{res.stderr}")
    if verbose and res.stderr.strip():
        print(res.stderr, file=sys.stderr)
    return obj


CALIB_SRC = os.path.join(PKG, "calib", "ceilings.hip")
CALIB_PATH = os.path.join(PKG, "libcoded_calib.so")


def build_calib(verbose: bool = False) -> str:
    """Compile the device-ceiling probes (calib/ceilings.hip) into their own library."""
    tmp = CALIB_PATH + ".tmp"
    # Matrix-instruction operands kept in vector registers: the rate probes'
    # accumulators are then not copied between register files every iteration.
    cmd = [hipcc(), "-x", "hip", *DEVICE, "-mllvm", "-amdgpu-mfma-vgpr-form=1", *COMMON, "-shared", CALIB_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compiling {CALIB_SRC} failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, CALIB_PATH)
    return CALIB_PATH


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(16, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"linking {LIB_NAME} failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB_PATH)
    build_calib(verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
