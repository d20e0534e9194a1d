"""Build libwsr.so (HIP kernels for gfx950 plus the C ABI) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT_DIR = os.path.join(PKG, "_build")
LIB_PATH = os.path.join(PKG, "libwsr.so")

ARCH = "gfx950"
COMMON = ["-O3", "-fPIC", "-std=c++17", "-Wall", f"-I{INCLUDE}", f"-I{CSRC}"]
# Packed fp32 instructions are kept out of every kernel (the host pass warns it does not know the
# feature; that is expected).
# The atomic optimizer turns a single-lane atomic with a return value into a wave-wide scan that
# consumes the result at once; the sweep's tile claims are issued ahead of use and must stay plain.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-ffp-contract=fast", "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    k_obj = os.path.join(OUT_DIR, "wsr_kernels.o")
    a_obj = os.path.join(OUT_DIR, "wsr_api.o")
    _run(["hipcc", *COMMON, *DEVICE, "-c", os.path.join(CSRC, "wsr_kernels.hip"), "-o", k_obj])
    _run(["hipcc", *COMMON, "-c", os.path.join(CSRC, "wsr_api.cpp"), "-o", a_obj])
    tmp = LIB_PATH + ".tmp"
    _run(["hipcc", "-shared", "-fPIC", f"--offload-arch={ARCH}", k_obj, a_obj, "-o", tmp])
    os.replace(tmp, LIB_PATH)
    if verbose:
        print("built", LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
