"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

Only draws numbers and encodes them into storage formats; none of the method's arithmetic lives
here.  Every value is a pure function of (seed, stream, element index), so any row of any tensor
can be regenerated on its own (the C source states the generator and distributions).

Storage conventions produced here (and consumed by both the oracle and the GPU library):
  * fp16 / bf16 tensors are returned as uint16 bit patterns;
  * a (M, K) matrix is row-major, element (i, k) is stream element i*K + k;
  * packed signed int4: uint8 (M, K/2), byte j of a row holds element 2j in the low nibble;
  * q4 block scales: fp16 bits (M, K/32), scale (i, b) is stream element i*(K/32) + b.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsynth.so")
SRC_PATH = os.path.join(_HERE, "synth.c")

F16, BF16 = 1, 2
# int8 row scales ~ U[2.5e-4, 1e-3): the scale max|w| / 127 of a symmetric int8 quantisation of an
# N(0, 0.02) row of a few thousand weights (max |w| about 4 sigma) is about 6e-4.
I8_SCALE_LO, I8_SCALE_HI = 2.5e-4, 1e-3
_FMT = {"f16": F16, "bf16": BF16, F16: F16, BF16: BF16}


DEV_LIB_PATH = os.path.join(_HERE, "libsynth_dev.so")
DEV_SRC_PATH = os.path.join(_HERE, "synth_dev.hip")


def build() -> str:
    """Compile libsynth.so (host) and libsynth_dev.so (the same generator for gfx950)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-fopenmp",
           SRC_PATH, "-o", LIB_PATH + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    cmd = ["hipcc", "-O3", "-fPIC", "-shared", "--offload-arch=gfx950", "-ffp-contract=off",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           DEV_SRC_PATH, "-o", DEV_LIB_PATH + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building {DEV_SRC_PATH} failed:\n{r.stderr}")
    os.replace(DEV_LIB_PATH + ".tmp", DEV_LIB_PATH)
    return LIB_PATH


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        u64, i64, i32, dbl, vp = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_int,
                                  ctypes.c_double, ctypes.c_void_p)
        L.synth_u64.argtypes = [u64, u64, u64]
        L.synth_u64.restype = u64
        L.synth_enc_f16.argtypes = [dbl]
        L.synth_enc_f16.restype = ctypes.c_uint16
        L.synth_enc_bf16.argtypes = [dbl]
        L.synth_enc_bf16.restype = ctypes.c_uint16
        L.synth_grid.argtypes = [u64, u64, u64]
        L.synth_grid.restype = ctypes.c_float
        L.synth_int4.argtypes = [u64, u64, u64]
        L.synth_int4.restype = i32
        L.synth_int8.argtypes = [u64, u64, u64]
        L.synth_int8.restype = i32
        L.synth_i8.argtypes = [vp, i64, u64, u64, u64, i32]
        L.synth_table_bytes.argtypes = []
        L.synth_table_bytes.restype = ctypes.c_size_t
        L.synth_table_build.argtypes = [vp, i32, dbl]
        L.synth_table_build.restype = i32
        L.synth_normal16.argtypes = [vp, i64, u64, u64, u64, vp, i32]
        L.synth_normal16_one.argtypes = [vp, u64, u64, u64]
        L.synth_normal16_one.restype = ctypes.c_uint16
        L.synth_grid_f32.argtypes = [vp, i64, u64, u64, u64, i32]
        L.synth_q4.argtypes = [vp, i64, u64, u64, u64, i32]
        L.synth_uniform16.argtypes = [vp, i64, u64, u64, u64, dbl, dbl, i32, i32]
        L.synth_encode16.argtypes = [vp, vp, i64, i32]
        for f in ("synth_normal16", "synth_grid_f32", "synth_q4", "synth_i8",
                  "synth_uniform16", "synth_encode16"):
            getattr(L, f).restype = None
        _lib = L
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _out(out, shape, dtype):
    if out is None:
        return np.empty(shape, dtype=dtype)
    assert out.dtype == dtype and out.flags.c_contiguous and out.size == int(np.prod(shape))
    return out


_tables = {}


def table(fmt, sigma) -> np.ndarray:
    """Sampling table of RNE(sigma * N(0, 1)) in fp16/bf16 (raw bytes of the C struct, cached)."""
    key = (_FMT[fmt], float(sigma))
    if key not in _tables:
        t = np.zeros(lib().synth_table_bytes(), dtype=np.uint8)
        if lib().synth_table_build(t.ctypes.data, key[0], key[1]) != 0:
            raise ValueError(f"cannot build a sampling table for sigma={sigma}")
        _tables[key] = t
    return _tables[key]


def table_arrays(fmt, sigma):
    """(accept thresholds uint64[65536], alias codes uint16[65536]) of the sampling table."""
    t = table(fmt, sigma)
    return t[: 8 * 65536].view(np.uint64), t[8 * 65536: 8 * 65536 + 2 * 65536].view(np.uint16)


def normal16(shape, sigma, fmt, seed=0, stream=0, e0=0, out=None, threads=None):
    """Codes of RNE(sigma * N(0,1)) in fp16/bf16 (uint16); flat element e0 + i of the stream."""
    a = _out(out, shape, np.uint16)
    lib().synth_normal16(a.ctypes.data, a.size, seed, stream, e0, table(fmt, sigma).ctypes.data,
                         threads or default_threads())
    return a


def grid_f32(shape, seed=0, stream=0, e0=0, out=None, threads=None):
    """Uniform on [-1, 1) on the 2^-23 grid (sums of up to 2^29 values are exact in double)."""
    a = _out(out, shape, np.float32)
    lib().synth_grid_f32(a.ctypes.data, a.size, seed, stream, e0, threads or default_threads())
    return a


def q4_codes(M, K, seed=0, stream=0, row0=0, out=None, threads=None):
    """Packed signed int4 codes of rows [row0, row0 + M) of a (*, K) matrix, uint8 (M, K/2)."""
    assert K % 2 == 0
    a = _out(out, (M, K // 2), np.uint8)
    lib().synth_q4(a.ctypes.data, a.size, seed, stream, row0 * K, threads or default_threads())
    return a


def uniform16(shape, lo, hi, fmt, seed=0, stream=0, e0=0, out=None, threads=None):
    a = _out(out, shape, np.uint16)
    lib().synth_uniform16(a.ctypes.data, a.size, seed, stream, e0, float(lo), float(hi),
                          _FMT[fmt], threads or default_threads())
    return a


def q4_scales(M, K, lo=0.005, hi=0.02, seed=0, stream=0, row0=0, out=None, threads=None):
    """fp16 block scales of rows [row0, row0 + M) of a (*, K) q4 matrix, uint16 (M, K/32)."""
    assert K % 32 == 0
    nb = K // 32
    return uniform16((M, nb), lo, hi, F16, seed, stream, row0 * nb, out, threads)


def i8_codes(M, K, seed=0, stream=0, row0=0, out=None, threads=None):
    """Signed int8 codes of rows [row0, row0 + M) of a (*, K) matrix, int8 (M, K)."""
    a = _out(out, (M, K), np.int8)
    lib().synth_i8(a.ctypes.data, a.size, seed, stream, row0 * K, threads or default_threads())
    return a


def i8_scales(M, lo=I8_SCALE_LO, hi=I8_SCALE_HI, seed=0, stream=0, row0=0, out=None, threads=None):
    """fp16 row scales of rows [row0, row0 + M) of an int8 matrix, uint16 (M,)."""
    return uniform16((M,), lo, hi, F16, seed, stream, row0, out, threads)


def int8(seed, stream, e):
    return lib().synth_int8(seed, stream, e)


def encode16(values, fmt):
    """Round doubles to fp16/bf16 bits (nearest-even), e.g. for hand-made test inputs."""
    v = np.ascontiguousarray(values, dtype=np.float64)
    a = np.empty(v.shape, dtype=np.uint16)
    lib().synth_encode16(a.ctypes.data, v.ctypes.data, v.size, _FMT[fmt])
    return a


def u64(seed, stream, e):
    return lib().synth_u64(seed, stream, e)
