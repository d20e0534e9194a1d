"""Pins for the CPU oracle: checks against what the paper and the mathematics fix, not against the
oracle's own formulas.

Each pin takes an `oracle.Oracle` and raises AssertionError on a mismatch.  They run against the
default build (tests/test_oracle_pins.py) and against copies of oracle.c with a planted mistake
(tests/test_oracle_mutants.py), where at least one pin must fail.

Independent references used here: numpy's IEEE half conversion and float32 reinterpretation for the
exhaustive decoding tables, Python `struct`'s half format, exact rational arithmetic
(`fractions.Fraction`) for brute force, and closed forms (identity, unit vectors, constant and
antisymmetric fills, hand-worked integer examples).
"""
from __future__ import annotations

import math
import struct
from fractions import Fraction

import numpy as np

import synth

ALL16 = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)


def _f16_ref(codes: np.ndarray) -> np.ndarray:
    return codes.view(np.float16).astype(np.float64)


def _bf16_ref(codes: np.ndarray) -> np.ndarray:
    with np.errstate(invalid="ignore"):     # NaN payloads widen with a warning; values are fine
        return (codes.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _dec(codes: np.ndarray, fmt: str) -> np.ndarray:
    return _f16_ref(codes) if fmt == "f16" else _bf16_ref(codes)


def _same(a: float, b: float) -> bool:
    return (math.isnan(a) and math.isnan(b)) or a == b


# ---- decoding tables ------------------------------------------------------------------------------

def pin_f16_exhaustive(ora):
    ref = _f16_ref(ALL16)
    for c in range(1 << 16):
        got = ora.f16(c)
        assert _same(got, ref[c]), f"fp16 code {c:#06x}: {got!r} != {ref[c]!r}"
    # a second, independent decoder for a spread of codes: Python's struct half format
    for c in range(0, 1 << 16, 97):
        want = struct.unpack("<e", struct.pack("<H", c))[0]
        assert _same(ora.f16(c), want), f"fp16 code {c:#06x} vs struct"


def pin_bf16_exhaustive(ora):
    ref = _bf16_ref(ALL16)
    for c in range(1 << 16):
        got = ora.bf16(c)
        assert _same(got, ref[c]), f"bf16 code {c:#06x}: {got!r} != {ref[c]!r}"


INT4_TABLE = {0: 0, 1: 1, 2: 2, 3: 3, 4: 4, 5: 5, 6: 6, 7: 7,
              8: -8, 9: -7, 10: -6, 11: -5, 12: -4, 13: -3, 14: -2, 15: -1}

# byte -> (element 2j, element 2j + 1): low nibble first
BYTE_TABLE = {0x08: (-8, 0), 0x7F: (-1, 7), 0xF0: (0, -1), 0x1F: (-1, 1), 0x80: (0, -8),
              0x00: (0, 0), 0xFF: (-1, -1), 0x97: (7, -7)}


def pin_int4_table(ora):
    for code, want in INT4_TABLE.items():
        assert ora.int4(code) == want, f"int4 code {code}"


def pin_q4_byte_table(ora):
    one = synth.encode16([1.0], "f16")[0]
    bytes_ = np.array(list(BYTE_TABLE), dtype=np.uint8)
    M, K = len(bytes_), 32
    Wq = np.zeros((M, K // 2), dtype=np.uint8)
    Wq[:, 5] = bytes_                       # elements 10 and 11 of each row
    S = np.full((M, 1), one, dtype=np.uint16)
    w = ora.dequant_q4(Wq, S)
    for r, b in enumerate(bytes_):
        lo, hi = BYTE_TABLE[int(b)]
        assert w[r, 10] == lo and w[r, 11] == hi, f"byte {b:#04x}: {w[r, 10:12]}"
        assert np.count_nonzero(w[r]) == (lo != 0) + (hi != 0)


# ---- probe ----------------------------------------------------------------------------------------

def pin_probe_closed_forms(ora):
    assert ora.probe_sum(np.full(1000, 0.375, np.float32)) == 375.0
    assert ora.probe_sum(np.full(4097, -1.0, np.float32)) == -4097.0
    assert ora.probe_sum(np.zeros(0, np.float32)) == 0.0
    assert ora.probe_sum(np.array([2.5], np.float32)) == 2.5
    # antisymmetric fill: x[i] = -x[n-1-i] sums to exactly zero (grid values, exact in double)
    half = synth.grid_f32(2048, seed=3, stream=9)
    x = np.concatenate([half, -half[::-1]])
    assert ora.probe_sum(x) == 0.0
    # odd length with a middle zero
    x = np.concatenate([half[:7], [0.0], -half[:7][::-1]]).astype(np.float32)
    assert ora.probe_sum(x) == 0.0


def pin_probe_brute_force(ora):
    # grid values: the double sum is exact in any order, so it equals the rational sum exactly
    x = synth.grid_f32(4096, seed=1, stream=5)
    exact = sum((Fraction(float(v)) for v in x), Fraction(0))
    assert ora.probe_sum(x) == float(exact)
    # general fp32 values (wide exponent range): within n * 2^-53 * sum|x| of the rational sum
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(3001) * np.exp2(rng.integers(-20, 20, 3001))).astype(np.float32)
    exact = sum((Fraction(float(v)) for v in x), Fraction(0))
    bound = len(x) * 2.0 ** -53 * float(np.abs(x.astype(np.float64)).sum())
    assert abs(ora.probe_sum(x) - float(exact)) <= bound


# ---- 16-bit GEMV -------------------------------------------------------------------------------------

def _rand16(shape, fmt, seed, stream, sigma=1.0):
    return synth.normal16(shape, sigma, fmt, seed=seed, stream=stream)


def pin_gemv16_hand(ora):
    # W = [[1, 2, 3], [4, 5, 6]], x = [1, -1, 2]  ->  y = [5, 11] (worked by hand)
    for fmt in ("f16", "bf16"):
        W = synth.encode16([[1, 2, 3], [4, 5, 6]], fmt)
        x = synth.encode16([1, -1, 2], fmt)
        assert list(ora.gemv16(W, x, fmt)) == [5.0, 11.0], fmt
    # a 3 x 2 example: [[0.5, -2], [3, 0.25], [-1, -1]] . [4, 8] = [-14, 14, -12]
    for fmt in ("f16", "bf16"):
        W = synth.encode16([[0.5, -2], [3, 0.25], [-1, -1]], fmt)
        x = synth.encode16([4, 8], fmt)
        assert list(ora.gemv16(W, x, fmt)) == [-14.0, 14.0, -12.0], fmt


def pin_gemv16_identity_and_units(ora):
    for fmt in ("f16", "bf16"):
        K = 48
        one, zero = synth.encode16([1.0, 0.0], fmt)
        eye = np.full((K, K), zero, np.uint16)
        np.fill_diagonal(eye, one)
        x = _rand16(K, fmt, 11, 1)
        assert np.array_equal(ora.gemv16(eye, x, fmt), _dec(x, fmt)), fmt
        M = 37
        W = _rand16((M, K), fmt, 11, 2, 0.02)
        for j in (0, 1, 17, K - 1):
            e = np.full(K, zero, np.uint16)
            e[j] = one
            assert np.array_equal(ora.gemv16(W, e, fmt), _dec(W[:, j], fmt)), (fmt, j)


def pin_gemv16_constant_forms(ora):
    for fmt in ("f16", "bf16"):
        M, K = 9, 40
        one = synth.encode16([1.0], fmt)[0]
        x = _rand16(K, fmt, 12, 1)
        W1 = np.full((M, K), one, np.uint16)
        sx = float(sum((Fraction(float(v)) for v in _dec(x, fmt)), Fraction(0)))
        y = ora.gemv16(W1, x, fmt)
        assert np.all(np.abs(y - sx) <= K * 2.0 ** -53 * np.abs(_dec(x, fmt)).sum()), fmt
        W = _rand16((M, K), fmt, 12, 2, 0.02)
        x1 = np.full(K, one, np.uint16)
        Wd = _dec(W, fmt)
        rows = [float(sum((Fraction(float(v)) for v in r), Fraction(0))) for r in Wd]
        y = ora.gemv16(W, x1, fmt)
        bound = K * 2.0 ** -53 * np.abs(Wd).sum(axis=1)
        assert np.all(np.abs(y - np.array(rows)) <= bound), fmt


def pin_gemv16_brute_force(ora):
    for fmt in ("f16", "bf16"):
        for (M, K, seed) in ((7, 24, 1), (13, 64, 2), (1, 5, 3), (64, 9, 4)):
            W = _rand16((M, K), fmt, seed, 3, 0.5)
            x = _rand16(K, fmt, seed, 4)
            Wd, xd = _dec(W, fmt), _dec(x, fmt)
            y = ora.gemv16(W, x, fmt)
            for i in range(M):
                exact = sum((Fraction(float(Wd[i, k])) * Fraction(float(xd[k])) for k in range(K)),
                            Fraction(0))
                bound = K * 2.0 ** -53 * float(np.abs(Wd[i] * xd).sum()) + 1e-300
                assert abs(y[i] - float(exact)) <= bound, (fmt, M, K, i)


def pin_gemv16_column_invariant(ora):
    # sum_i y_i == (column sums of W) . x, both sides exact rationals compared within rounding
    for fmt in ("f16", "bf16"):
        M, K = 33, 56
        W = _rand16((M, K), fmt, 21, 5, 0.02)
        x = _rand16(K, fmt, 21, 6)
        Wd, xd = _dec(W, fmt), _dec(x, fmt)
        col = [sum((Fraction(float(Wd[i, k])) for i in range(M)), Fraction(0)) for k in range(K)]
        rhs = float(sum((col[k] * Fraction(float(xd[k])) for k in range(K)), Fraction(0)))
        lhs = float(sum((Fraction(float(v)) for v in ora.gemv16(W, x, fmt)), Fraction(0)))
        bound = (M + K) * 2.0 ** -52 * float(np.abs(Wd * xd).sum())
        assert abs(lhs - rhs) <= bound, fmt


# ---- q4 -------------------------------------------------------------------------------------------

def _q4(M, K, seed, unit_scale=False):
    Wq = synth.q4_codes(M, K, seed=seed, stream=7)
    if unit_scale:
        S = np.full((M, K // 32), synth.encode16([1.0], "f16")[0], np.uint16)
    else:
        S = synth.q4_scales(M, K, seed=seed, stream=8)
    return Wq, S


def _q4_ref(Wq, S):
    """Independent decode: numpy nibble split, hand table, numpy fp16."""
    M, K = Wq.shape[0], Wq.shape[1] * 2
    codes = np.empty((M, K), np.int64)
    codes[:, 0::2] = Wq & 0xF
    codes[:, 1::2] = Wq >> 4
    q = np.vectorize(INT4_TABLE.get)(codes)
    s = np.repeat(_f16_ref(S), 32, axis=1)
    return q, s


def pin_q4_units(ora):
    M, K = 11, 96
    Wq, S = _q4(M, K, 31)
    q, s = _q4_ref(Wq, S)
    zero, one = synth.encode16([0.0, 1.0], "f16")
    for j in (0, 1, 2, 31, 32, 33, 63, 64, K - 1):
        e = np.full(K, zero, np.uint16)
        e[j] = one
        y = ora.gemv_q4(Wq, S, e)
        assert np.array_equal(y, q[:, j] * s[:, j]), j
    assert np.array_equal(ora.dequant_q4(Wq, S), q * s)


def pin_q4_identity_blocks(ora):
    K = 64
    one = synth.encode16([1.0], "f16")[0]
    Wq = np.zeros((K, K // 2), np.uint8)
    for i in range(K):                      # q[i, i] = 1
        Wq[i, i // 2] = 0x01 if i % 2 == 0 else 0x10
    S = np.full((K, K // 32), one, np.uint16)
    x = _rand16(K, "f16", 41, 1)
    assert np.array_equal(ora.gemv_q4(Wq, S, x), _f16_ref(x))


def pin_q4_brute_force(ora):
    for (M, K, seed) in ((5, 64, 1), (3, 160, 2), (17, 32, 3)):
        Wq, S = _q4(M, K, seed)
        x = _rand16(K, "f16", seed, 9)
        q, s = _q4_ref(Wq, S)
        xd = _f16_ref(x)
        y = ora.gemv_q4(Wq, S, x)
        for i in range(M):
            exact = sum((Fraction(int(q[i, k])) * Fraction(float(s[i, k])) * Fraction(float(xd[k]))
                         for k in range(K)), Fraction(0))
            bound = K * 2.0 ** -53 * float(np.abs(q[i] * s[i] * xd).sum()) + 1e-300
            assert abs(y[i] - float(exact)) <= bound, (M, K, i)


def pin_q4_column_invariant(ora):
    M, K = 21, 128
    Wq, S = _q4(M, K, 51)
    x = _rand16(K, "f16", 51, 2)
    q, s = _q4_ref(Wq, S)
    w, xd = q * s, _f16_ref(x)
    col = [sum((Fraction(float(w[i, k])) for i in range(M)), Fraction(0)) for k in range(K)]
    rhs = float(sum((col[k] * Fraction(float(xd[k])) for k in range(K)), Fraction(0)))
    lhs = float(sum((Fraction(float(v)) for v in ora.gemv_q4(Wq, S, x)), Fraction(0)))
    assert abs(lhs - rhs) <= (M + K) * 2.0 ** -52 * float(np.abs(w * xd).sum())


# ---- int8 with fp16 row scales ----------------------------------------------------------------------

def pin_int8_table(ora):
    """All 256 bytes against numpy's two's-complement reinterpretation."""
    ref = np.arange(256, dtype=np.uint16).astype(np.uint8).view(np.int8)
    for b in range(256):
        assert ora.int8(b) == int(ref[b]), f"byte {b:#04x}"


def _i8(M, K, seed):
    return synth.i8_codes(M, K, seed=seed, stream=21), synth.i8_scales(M, seed=seed, stream=22)


def pin_i8_units(ora):
    M, K = 13, 80
    Wq, S = _i8(M, K, 81)
    q, s = Wq.astype(np.float64), _f16_ref(S)
    zero, one = synth.encode16([0.0, 1.0], "f16")
    for j in (0, 1, 15, 16, 17, 63, K - 1):
        e = np.full(K, zero, np.uint16)
        e[j] = one
        assert np.array_equal(ora.gemv_i8(Wq, S, e), q[:, j] * s), j
    assert ora.i8_weight(Wq, S, 3, 7) == q[3, 7] * s[3]


def pin_i8_row_scales(ora):
    """Every weight 1 and distinct scales per row: y_i = s_i * sum(x), exactly in rationals."""
    M, K = 9, 48
    Wq = np.ones((M, K), np.int8)
    S = synth.encode16([0.5 + 0.125 * i for i in range(M)], "f16")
    x = _rand16(K, "f16", 82, 3)
    xs = sum((Fraction(float(v)) for v in _f16_ref(x)), Fraction(0))
    y = ora.gemv_i8(Wq, S, x)
    for i in range(M):
        assert abs(y[i] - float(Fraction(float(_f16_ref(S)[i])) * xs)) <= K * 2.0 ** -50, i


def pin_i8_brute_force(ora):
    for (M, K, seed) in ((4, 48, 1), (7, 16, 2), (3, 112, 3)):
        Wq, S = _i8(M, K, 83 + seed)
        x = _rand16(K, "f16", seed, 19)
        q, s, xd = Wq.astype(np.int64), _f16_ref(S), _f16_ref(x)
        y = ora.gemv_i8(Wq, S, x)
        for i in range(M):
            exact = sum((Fraction(int(q[i, k])) * Fraction(float(s[i])) * Fraction(float(xd[k]))
                         for k in range(K)), Fraction(0))
            bound = K * 2.0 ** -53 * float(np.abs(q[i] * s[i] * xd).sum()) + 1e-300
            assert abs(y[i] - float(exact)) <= bound, (M, K, i)


def pin_i8_column_invariant(ora):
    M, K = 19, 64
    Wq, S = _i8(M, K, 87)
    x = _rand16(K, "f16", 87, 2)
    w, xd = Wq.astype(np.float64) * _f16_ref(S)[:, None], _f16_ref(x)
    col = [sum((Fraction(float(w[i, k])) for i in range(M)), Fraction(0)) for k in range(K)]
    rhs = float(sum((col[k] * Fraction(float(xd[k])) for k in range(K)), Fraction(0)))
    lhs = float(sum((Fraction(float(v)) for v in ora.gemv_i8(Wq, S, x)), Fraction(0)))
    assert abs(lhs - rhs) <= (M + K) * 2.0 ** -52 * float(np.abs(w * xd).sum())


# ---- decode sweep ----------------------------------------------------------------------------------

def pin_sweep_tokens_and_order(ora):
    """Two tiny layers plus a head, three tokens, mixed formats: every (token, matrix) output equals
    the exact rational product of that matrix with that token's activation."""
    shapes = [("bf16", 6, 16), ("bf16", 4, 16), ("q4", 5, 64), ("i8", 3, 32), ("f16", 3, 24)]
    mats, xs = [], []
    for m, (fmt, M, K) in enumerate(shapes):
        if fmt == "q4":
            Wq, S = _q4(M, K, 60 + m)
            mats.append({"fmt": fmt, "w": Wq, "s": S})
            q, s = _q4_ref(Wq, S)
            dense = q * s
            xfmt = "f16"
        elif fmt == "i8":
            Wq, S = _i8(M, K, 60 + m)
            mats.append({"fmt": fmt, "w": Wq, "s": S})
            dense = Wq.astype(np.float64) * _f16_ref(S)[:, None]
            xfmt = "f16"
        else:
            W = _rand16((M, K), fmt, 60 + m, 1, 0.25)
            mats.append({"fmt": fmt, "w": W})
            dense = _dec(W, fmt)
            xfmt = fmt
        xs.append([_rand16(K, xfmt, 70 + m, 100 + t) for t in range(3)])
        mats[-1]["dense"], mats[-1]["xfmt"] = dense, xfmt
    out = ora.sweep(mats, xs, range(3))
    assert sorted(out) == [(t, m) for t in range(3) for m in range(len(shapes))]
    for (t, m), y in out.items():
        dense, xd = mats[m]["dense"], _dec(xs[m][t], mats[m]["xfmt"])
        for i in range(dense.shape[0]):
            exact = sum((Fraction(float(dense[i, k])) * Fraction(float(xd[k]))
                         for k in range(dense.shape[1])), Fraction(0))
            bound = dense.shape[1] * 2.0 ** -53 * float(np.abs(dense[i] * xd).sum()) + 1e-300
            assert abs(y[i] - float(exact)) <= bound, (t, m, i)


ALL_PINS = [v for k, v in dict(globals()).items() if k.startswith("pin_")]
