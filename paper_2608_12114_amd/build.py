"""Build libwsr.so (HIP kernels for gfx950 plus the C ABI) in-tree with hipcc."""
from __future__ import annotations

import collections
import os
import re
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
# Matrix instructions write ordinary vector registers (not the accumulation registers), so their
# results are scaled and summed without a copy out first.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-ffp-contract=fast", "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
          "-mllvm", "-amdgpu-mfma-vgpr-form"]


# A toolchain hazard checked on every build.  The AMDGPU backend's pre-emit peephole deletes an
# `s_and_b64 vcc, vcc, exec` after a vector compare when a VCC branch follows, without checking
# whether a scalar select still reads the SCC that instruction defines; the select then takes a
# stale condition.  It turned a row clamp min(r0 + R, M) into r0 + R, so a kernel read and wrote
# rows past the end of its matrix.  The compile prints the machine code just before and after that
# pass (printing does not change code generation), and the build fails if the pass removed any
# instruction whose SCC definition was live.
_PEEPHOLE = "si-pre-emit-peephole"
_MIR_FLAGS = ["-mllvm", f"-print-before={_PEEPHOLE}", "-mllvm", f"-print-after={_PEEPHOLE}"]


def dropped_live_scc(dump: str) -> list[str]:
    """Instructions with a live SCC definition present before the pass and gone after it."""
    parts = re.split(r"^# \*\*\* IR Dump (Before|After) [^\n]*\n", dump, flags=re.M)
    seen: dict[str, dict[str, collections.Counter]] = {}
    for kind, body in zip(parts[1::2], parts[2::2]):
        m = re.search(r"^# Machine code for function (\S+?):", body, re.M)
        if not m:
            continue
        live = collections.Counter(l.strip() for l in body.splitlines() if "implicit-def $scc" in l)
        seen.setdefault(m.group(1), {})[kind] = live
    out = []
    for fn, d in seen.items():
        for line, n in (d.get("Before", collections.Counter()) - d.get("After", collections.Counter())).items():
            out.append(f"{fn}: {line} (x{n})")
    return out


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}")
    return r


KERNEL_FILES = ("wsr_kernels.hip", "wsr_mma.hip", "wsr_copy.hip")


def _compile_kernels(src: str) -> str:
    obj = os.path.join(OUT_DIR, src.replace(".hip", ".o"))
    r = _run(["hipcc", *COMMON, *DEVICE, *_MIR_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
    if "IR Dump Before" not in r.stderr:
        raise RuntimeError(f"build: the compiler printed no machine code for the peephole check ({src})")
    dropped = dropped_live_scc(r.stderr)
    if dropped:
        raise RuntimeError(f"build: the pre-emit peephole removed live SCC definitions in {src} "
                           "(miscompiled selects):\n  " + "\n  ".join(dropped))
    return obj


def _compile_api() -> str:
    obj = os.path.join(OUT_DIR, "wsr_api.o")
    _run(["hipcc", *COMMON, "-c", os.path.join(CSRC, "wsr_api.cpp"), "-o", obj])
    return obj


def build(verbose: bool = False) -> str:
    """Compile the kernel files and the C ABI (each its own hipcc process, run side by side), then
    link libwsr.so and move it into place in one rename."""
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(OUT_DIR, exist_ok=True)
    with ThreadPoolExecutor(len(KERNEL_FILES) + 1) as ex:
        futs = [ex.submit(_compile_kernels, src) for src in KERNEL_FILES]
        api = ex.submit(_compile_api)
        objs = [f.result() for f in futs] + [api.result()]
    tmp = LIB_PATH + ".tmp"
    _run(["hipcc", "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp])
    os.replace(tmp, LIB_PATH)
    if verbose:
        print("built", LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
