"""int8 weights with fp16 row scales, the matched protocol's format (Sec. 3.1): the GEMV against
the oracle, exact dequantisation through unit vectors, the multi-column kernel bit for bit against
the single-column one, and decode sweeps holding int8 matrices (alone, mixed with q4 and 16-bit
matrices, batched) at small sizes and at the protocol's full 12 x 12288 x 7168 shape."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, sample_rows, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]


def gemv_i8(Wq, S, x, M, K):
    y = torch.full((max(M, 1),), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_i8(dv.to_device(Wq), dv.to_device(S), dv.to_device(x), y, M, K, stream())
    return y[:M].cpu().numpy()


def inputs(M, K, seed, s0):
    return (synth.i8_codes(M, K, seed=seed, stream=s0), synth.i8_scales(M, seed=seed, stream=s0 + 1),
            synth.normal16(K, wl.X_SIGMA, "f16", seed=seed, stream=s0 + 2))


# (3, 28672) once faulted the GPU: the GEMV's row clamp min(r0 + R, M) was miscompiled to r0 + R, so
# with 8-row groups a wave read 5 rows (140 KB) past the codes.  The kernel no longer clamps with a
# select, the build rejects the miscompile, and tests/test_gpu_bounds.py checks that only rows < M
# are written.
SHAPES = [(1, 16), (5, 32), (37, 2064), (300, 4096), (4096, 4096), (1024, 14336), (14336, 4096),
          (3, 28672), (12288, 7168)]


@pytest.mark.parametrize("M,K", SHAPES)
def test_gemv_i8_parity(M, K):
    Wq, S, x = inputs(M, K, 0, 401)
    y = gemv_i8(Wq, S, x, M, K)
    assert rel_l2(y, oracle.get().gemv_i8(Wq, S, x, threads=8)) <= TOL
    assert np.array_equal(f32_bits(y), f32_bits(gemv_i8(Wq, S, x, M, K)))


def test_gemv_i8_empty():
    # M = 0: nothing is written
    y = torch.full((4,), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_i8(None, None, None, y, 0, 16, stream())
    torch.cuda.synchronize()
    assert np.isnan(y.cpu().numpy()).all()
    # K = 0: every output is the empty sum (codes and activations are never read)
    y = torch.full((5,), 7.0, device="cuda")
    s = dv.to_device(synth.i8_scales(5, seed=1, stream=407))
    wsr.wsr_gemv_i8(y, s, y, y, 5, 0, stream())
    assert y.cpu().tolist() == [0.0] * 5


def test_gemv_i8_dequant_exact_via_unit_vectors():
    """x = e_j returns column j of the dequantised matrix, q * s, bit for bit in fp32 (q * s needs
    at most 19 significant bits)."""
    M, K = 259, 4112
    Wq = synth.i8_codes(M, K, seed=3, stream=404)
    S = synth.i8_scales(M, seed=3, stream=405)
    ora = oracle.get()
    zero, one = synth.encode16([0.0, 1.0], "f16")
    for j in (0, 1, 2, 3, 7, 8, 15, 16, 17, 1023, 1024, 2047, 4095, K - 1):
        e = np.full(K, zero, np.uint16)
        e[j] = one
        want = np.array([ora.i8_weight(Wq, S, i, j) for i in range(M)])
        assert np.array_equal(f32_bits(gemv_i8(Wq, S, e, M, K)), f32_bits(want)), j


def test_gemv_i8_extreme_codes():
    """Rows of all -128, all 127 and alternating extremes against large activations: the decode's
    code offset (128 per element) and its removal stay within the parity bound."""
    K = 4096
    rows = [np.full(K, -128, np.int8), np.full(K, 127, np.int8),
            np.where(np.arange(K) % 2 == 0, -128, 127).astype(np.int8), np.zeros(K, np.int8)]
    Wq = np.stack(rows)
    S = synth.encode16([1e-3, 2.5e-4, 5e-4, 1e-3], "f16")
    for sigma in (1.0, 300.0):
        x = synth.normal16(K, sigma, "f16", seed=5, stream=406)
        y = gemv_i8(Wq, S, x, 4, K)
        want = oracle.get().gemv_i8(Wq, S, x)
        assert y[3] == 0.0
        for i in range(3):
            assert abs(y[i] - want[i]) <= TOL * np.abs(want[:3]).max(), (sigma, i)


@pytest.mark.parametrize("T", [1, 2, 4, 8])
@pytest.mark.parametrize("M,K", [(37, 512), (258, 4096), (300, 14336), (5, 16), (9, 2064)])
def test_gemv_i8_cols_parity_and_bitwise(T, M, K):
    Wqh = synth.i8_codes(M, K, seed=6, stream=411)
    Sh = synth.i8_scales(M, seed=6, stream=412)
    Xh = synth.normal16((T, K), wl.X_SIGMA, "f16", seed=6, stream=413)
    Wq, S, X = dv.to_device(Wqh), dv.to_device(Sh), dv.to_device(Xh)
    Y = torch.full((T, M), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_i8_cols(Wq, S, X, K * 2, Y, M * 4, M, K, T, stream())
    Y = Y.cpu().numpy()
    ora = oracle.get()
    for t in range(T):
        assert rel_l2(Y[t], ora.gemv_i8(Wqh, Sh, Xh[t], threads=8)) <= TOL, t
        assert np.array_equal(f32_bits(Y[t]), f32_bits(gemv_i8(Wqh, Sh, Xh[t], M, K))), t


# ---- decode sweeps holding int8 matrices -------------------------------------------------------

def run(inp, tokens, batch=None):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(inp.specs())
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    if batch is None:
        wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())
    else:
        wsr.wsr_decode_sweep_batched(mats, tokens, batch, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


def oracle_y(inp, i, t, rows=None):
    ora = oracle.get()
    fmt, x = inp.fmts[i], inp.host_x(i, t)

    def one(hw, threads):
        if fmt in (wl.Q4, wl.I8):
            return ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x, threads)
        return ora.gemv16(hw, x, fmt, threads=threads)

    if rows is None:
        return one(inp.host_weights(i), 8)
    return np.array([one(inp.host_weights(i, int(r), 1), 1)[0] for r in rows])


@pytest.fixture(scope="module")
def model_i8():
    mats = wl.decode_matrices(dv.small_model(layers=3, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.I8, wl.Q4, wl.BF16, wl.I8)[m.layer] for m in mats]     # head (layer 3) int8
    return dv.SweepInputs(mats, fmts, tokens=11)


def test_sweep_with_i8_parity(model_i8):
    ys = run(model_i8, 11)
    for i, m in enumerate(model_i8.mats):
        for t in (0, 10):
            assert rel_l2(ys[i][t], oracle_y(model_i8, i, t)) <= TOL, (m.name, m.layer, t)


@pytest.mark.parametrize("batch", [2, 4, 8, 16])
def test_sweep_with_i8_batched_equals_sequential(model_i8, batch):
    """int8, q4 and bf16 matrices in one table; batch 16 runs as passes of 8."""
    seq = run(model_i8, 11)
    bat = run(model_i8, 11, batch)
    for a, b in zip(seq, bat):
        assert np.array_equal(f32_bits(a), f32_bits(b))


@pytest.mark.parametrize("M,K", [(1000, 2064), (1003, 4096), (517, 1024), (75, 7168)])
def test_sweep_i8_only_equals_gemv(M, K):
    """A table of int8 matrices only (the uniform int8 sweep kernel) reproduces wsr_gemv_i8 bit
    for bit, matrix by matrix: rows of whole 64-chunk steps (K a multiple of 1024) take the
    pipelined row loop, across row groups and with ragged row counts, the others the plain one."""
    mats = wl.protocol_matrices(n=5, M=M, K=K)
    inp = dv.SweepInputs(mats, [wl.I8] * len(mats), tokens=2)
    ys = run(inp, 2)
    for i, m in enumerate(mats):
        Wq, S = inp.host_weights(i)
        for t in range(2):
            assert np.array_equal(f32_bits(ys[i][t]), f32_bits(gemv_i8(Wq, S, inp.host_x(i, t), m.M, m.K))), (i, t)


def test_protocol_full_size():
    """The protocol pass at its full shape (12 matrices of 12288 x 7168, int8 with row scales), in
    the launch configuration the benchmark times: batch-1 sweep and a batch of 8, every matrix
    checked on sampled rows."""
    mats = wl.protocol_matrices()
    inp = dv.SweepInputs(mats, [wl.I8] * len(mats), tokens=8)
    assert inp.weight_bytes() == wl.PROTOCOL_MATRICES * (wl.PROTOCOL_M * wl.PROTOCOL_K + wl.PROTOCOL_M * 2)
    seq = run(inp, 8)
    bat = run(inp, 8, 8)
    for i, m in enumerate(mats):
        assert np.array_equal(f32_bits(seq[i]), f32_bits(bat[i])), i
        rows = sample_rows(m.M, n=8, seed=i)
        for t in (0, 7):
            assert rel_l2(seq[i][t][rows], oracle_y(inp, i, t, rows)) <= TOL, (i, t)
    del inp
    torch.cuda.empty_cache()
