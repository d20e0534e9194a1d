"""CPU oracle for the weight-streaming read path - TEST INFRASTRUCTURE ONLY.

Only `tests/`, `__graft_entry__.smoke()` and the `cpu_baseline` leg of `bench.py` may import this
package.  The GPU library and its binding never do, and share no code with it.

The arithmetic lives in `oracle.c` (plain C, every value decoded to double, every sum in double in
ascending index order).  This module only marshals numpy arrays into it, plus the decode sweep,
which is the GEMV definition applied to every matrix of every token in order:

    for t in tokens:  for m in matrices (layer order):  y_m(t) = W_m . x_m(t)

(paper Sec. 6.2: a batch-1 token reads every weight once; Sec. 3.1: one pass visits every matrix).

Pins (tests/test_oracle_pins.py): exhaustive fp16 / bf16 / int4 decoding against independent
libraries and a hand table, exact closed forms (identity, unit vectors, constant fills, antisymmetric
fills), the column-sum invariant, exact rational brute force on small shapes, and mutation checks that
plant plausible mistakes in a copy of oracle.c and require the pins to catch each one.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")
CFLAGS = ["-O2", "-ffp-contract=off", "-fPIC", "-shared", "-fopenmp"]

F16, BF16 = 1, 2
_FMT = {"f16": F16, "bf16": BF16, F16: F16, BF16: BF16}


def build(src: str = SRC_PATH, out: str = LIB_PATH) -> str:
    """Compile the oracle (host gcc; no fast-math, no FMA contraction)."""
    subprocess.run(["gcc", *CFLAGS, src, "-o", out + ".tmp", "-lm"], check=True)
    os.replace(out + ".tmp", out)
    return out


def _bind(L: ctypes.CDLL) -> ctypes.CDLL:
    i64, i32, dbl, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_void_p
    L.ora_f16_to_f64.argtypes = [ctypes.c_uint16]
    L.ora_f16_to_f64.restype = dbl
    L.ora_bf16_to_f64.argtypes = [ctypes.c_uint16]
    L.ora_bf16_to_f64.restype = dbl
    L.ora_int4.argtypes = [ctypes.c_uint]
    L.ora_int4.restype = i32
    L.ora_probe_sum.argtypes = [vp, i64]
    L.ora_probe_sum.restype = dbl
    L.ora_gemv16.argtypes = [vp, vp, i64, i64, i32, vp, i32]
    L.ora_gemv16.restype = None
    L.ora_q4_weight.argtypes = [vp, vp, i64, i64, i64]
    L.ora_q4_weight.restype = dbl
    L.ora_dequant_q4.argtypes = [vp, vp, i64, i64, vp]
    L.ora_dequant_q4.restype = None
    L.ora_gemv_q4.argtypes = [vp, vp, vp, i64, i64, vp, i32]
    L.ora_gemv_q4.restype = None
    L.ora_int8.argtypes = [ctypes.c_uint]
    L.ora_int8.restype = i32
    L.ora_i8_weight.argtypes = [vp, vp, i64, i64, i64]
    L.ora_i8_weight.restype = dbl
    L.ora_gemv_i8.argtypes = [vp, vp, vp, i64, i64, vp, i32]
    L.ora_gemv_i8.restype = None
    return L


class Oracle:
    """numpy front end over one build of oracle.c (the default build, or a test's own copy)."""

    def __init__(self, lib_path: str = LIB_PATH):
        if lib_path == LIB_PATH and not os.path.exists(LIB_PATH):
            build()
        self.L = _bind(ctypes.CDLL(lib_path))

    # -- decoders --
    def f16(self, code: int) -> float:
        return self.L.ora_f16_to_f64(code)

    def bf16(self, code: int) -> float:
        return self.L.ora_bf16_to_f64(code)

    def int4(self, code: int) -> int:
        return self.L.ora_int4(code)

    # -- probe --
    def probe_sum(self, buf: np.ndarray) -> float:
        b = np.ascontiguousarray(buf, dtype=np.float32)
        return self.L.ora_probe_sum(b.ctypes.data, b.size)

    # -- GEMVs --
    def gemv16(self, W: np.ndarray, x: np.ndarray, fmt, threads: int = 1) -> np.ndarray:
        W = np.ascontiguousarray(W, dtype=np.uint16)
        x = np.ascontiguousarray(x, dtype=np.uint16)
        M, K = W.shape
        assert x.shape == (K,)
        y = np.empty(M, dtype=np.float64)
        self.L.ora_gemv16(W.ctypes.data, x.ctypes.data, M, K, _FMT[fmt], y.ctypes.data, threads)
        return y

    def dequant_q4(self, Wq: np.ndarray, S: np.ndarray) -> np.ndarray:
        Wq = np.ascontiguousarray(Wq, dtype=np.uint8)
        S = np.ascontiguousarray(S, dtype=np.uint16)
        M, K = Wq.shape[0], Wq.shape[1] * 2
        assert S.shape == (M, K // 32)
        w = np.empty((M, K), dtype=np.float64)
        self.L.ora_dequant_q4(Wq.ctypes.data, S.ctypes.data, M, K, w.ctypes.data)
        return w

    def int8(self, byte: int) -> int:
        return self.L.ora_int8(byte)

    def i8_weight(self, Wq: np.ndarray, S: np.ndarray, i: int, k: int) -> float:
        Wq = np.ascontiguousarray(Wq).view(np.uint8)
        S = np.ascontiguousarray(S, dtype=np.uint16)
        return self.L.ora_i8_weight(Wq.ctypes.data, S.ctypes.data, Wq.shape[1], i, k)

    def gemv_i8(self, Wq: np.ndarray, S: np.ndarray, x: np.ndarray, threads: int = 1) -> np.ndarray:
        Wq = np.ascontiguousarray(Wq).view(np.uint8)
        S = np.ascontiguousarray(S, dtype=np.uint16)
        x = np.ascontiguousarray(x, dtype=np.uint16)
        M, K = Wq.shape
        assert S.shape == (M,) and x.shape == (K,)
        y = np.empty(M, dtype=np.float64)
        self.L.ora_gemv_i8(Wq.ctypes.data, S.ctypes.data, x.ctypes.data, M, K, y.ctypes.data, threads)
        return y

    def gemv_q4(self, Wq: np.ndarray, S: np.ndarray, x: np.ndarray, threads: int = 1) -> np.ndarray:
        Wq = np.ascontiguousarray(Wq, dtype=np.uint8)
        S = np.ascontiguousarray(S, dtype=np.uint16)
        x = np.ascontiguousarray(x, dtype=np.uint16)
        M, K = Wq.shape[0], Wq.shape[1] * 2
        assert S.shape == (M, K // 32) and x.shape == (K,)
        y = np.empty(M, dtype=np.float64)
        self.L.ora_gemv_q4(Wq.ctypes.data, S.ctypes.data, x.ctypes.data, M, K, y.ctypes.data,
                           threads)
        return y

    def gemv(self, mat: dict, x: np.ndarray, threads: int = 1) -> np.ndarray:
        """GEMV of one sweep matrix: mat = {"fmt": "f16"|"bf16"|"q4"|"i8", "w": ..., "s": ...}."""
        if mat["fmt"] == "q4":
            return self.gemv_q4(mat["w"], mat["s"], x, threads)
        if mat["fmt"] == "i8":
            return self.gemv_i8(mat["w"], mat["s"], x, threads)
        return self.gemv16(mat["w"], x, mat["fmt"], threads)

    # -- decode sweep --
    def sweep(self, mats: list, xs: list, tokens, threads: int = 1) -> dict:
        """y[(t, m)] = W_m . x_m(t) for every token t and matrix m, in that order.

        mats[m]: dict as in gemv(); xs[m][t]: activation vector of matrix m at token t.
        """
        out = {}
        for t in tokens:
            for m, mat in enumerate(mats):
                out[(t, m)] = self.gemv(mat, xs[m][t], threads)
        return out


_default = None


def get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
