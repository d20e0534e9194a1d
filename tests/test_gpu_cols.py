"""Several activation columns per weight read (the multi-column kernel of Sec. 3.4 and 5.2): every
column must match the oracle within 2e-3 and equal the single-column result bit for bit, and a
batched decode sweep must reproduce the token-by-token sweep bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]
FMT = {"f16": wsr.WSR_F16, "bf16": wsr.WSR_BF16}


def single(W, x, fmt, M, K):
    y = torch.full((max(M, 1),), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_f16(W, x, y, M, K, FMT[fmt], stream())
    return y[:M].cpu().numpy()


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
@pytest.mark.parametrize("T", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("M,K", [(37, 520), (258, 4096), (1000, 14336), (5, 8)])
def test_cols_parity_and_bitwise(fmt, T, M, K):
    Wh = synth.normal16((M, K), wl.W_SIGMA, fmt, seed=3, stream=301)
    Xh = synth.normal16((T, K), wl.X_SIGMA, fmt, seed=3, stream=302)
    W, X = dv.to_device(Wh), dv.to_device(Xh)
    Y = torch.full((T, M), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_f16_cols(W, X, K * 2, Y, M * 4, M, K, T, FMT[fmt], stream())
    Y = Y.cpu().numpy()
    ora = oracle.get()
    for t in range(T):
        assert rel_l2(Y[t], ora.gemv16(Wh, Xh[t], fmt, threads=8)) <= TOL, t
        assert np.array_equal(f32_bits(Y[t]), f32_bits(single(W, X[t], fmt, M, K))), t


@pytest.mark.parametrize("T", [2, 16])
def test_cols_strides(T):
    """A zero activation stride (every column reads one x) and output columns with gaps: the gaps
    stay untouched."""
    M, K, gap = 300, 1024, 7
    Wh = synth.normal16((M, K), wl.W_SIGMA, "bf16", seed=4, stream=303)
    xh = synth.normal16(K, wl.X_SIGMA, "bf16", seed=4, stream=304)
    W, x = dv.to_device(Wh), dv.to_device(xh)
    ys = M + gap
    Y = torch.full((T, ys), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_f16_cols(W, x, 0, Y, ys * 4, M, K, T, wsr.WSR_BF16, stream())
    Y = Y.cpu().numpy()
    ref = single(W, x, "bf16", M, K)
    for t in range(T):
        assert np.array_equal(f32_bits(Y[t, :M]), f32_bits(ref)), t
        assert np.isnan(Y[t, M:]).all(), t


def run(inp, tokens, batch, chained=False):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(inp.specs(chained=chained))
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    if batch is None:
        wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())
    else:
        wsr.wsr_decode_sweep_batched(mats, tokens, batch, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


@pytest.fixture(scope="module")
def model16():
    mats = wl.decode_matrices(dv.small_model(layers=2, d=512, ffn=1536, vocab=3000))
    fmts = [("bf16", "f16", "bf16")[m.layer] for m in mats]
    return dv.SweepInputs(mats, fmts, tokens=21)


@pytest.mark.parametrize("batch", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("chained", [False, True])
def test_batched_sweep_equals_sequential(model16, batch, chained):
    """21 tokens: full passes of `batch` tokens, then the rest in smaller passes."""
    seq = run(model16, 21, None, chained)
    bat = run(model16, 21, batch, chained)
    for a, b in zip(seq, bat):
        assert np.array_equal(f32_bits(a), f32_bits(b))


def test_batched_sweep_parity(model16):
    ys = run(model16, 21, 16)
    ora = oracle.get()
    for i, (m, fmt) in enumerate(zip(model16.mats, model16.fmts)):
        for t in (0, 15, 20):
            want = ora.gemv16(model16.host_weights(i), model16.host_x(i, t), fmt, threads=8)
            assert rel_l2(ys[i][t], want) <= TOL, (m.name, m.layer, t)


def single_q4(Wq, S, x, M, K):
    y = torch.full((max(M, 1),), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_q4(Wq, S, x, y, M, K, stream())
    return y[:M].cpu().numpy()


@pytest.mark.parametrize("T", [1, 2, 4, 8])
@pytest.mark.parametrize("M,K", [(37, 512), (258, 4096), (300, 14336), (5, 32), (9, 2080)])
def test_q4_cols_parity_and_bitwise(T, M, K):
    Wqh = synth.q4_codes(M, K, seed=5, stream=311)
    Sh = synth.q4_scales(M, K, seed=5, stream=312)
    Xh = synth.normal16((T, K), wl.X_SIGMA, "f16", seed=5, stream=313)
    Wq, S, X = dv.to_device(Wqh), dv.to_device(Sh), dv.to_device(Xh)
    Y = torch.full((T, M), float("nan"), dtype=torch.float32, device="cuda")
    wsr.wsr_gemv_q4_cols(Wq, S, X, K * 2, Y, M * 4, M, K, T, stream())
    Y = Y.cpu().numpy()
    ora = oracle.get()
    for t in range(T):
        assert rel_l2(Y[t], ora.gemv_q4(Wqh, Sh, Xh[t], threads=8)) <= TOL, t
        assert np.array_equal(f32_bits(Y[t]), f32_bits(single_q4(Wq, S, X[t], M, K))), t


@pytest.fixture(scope="module")
def model_mixed():
    mats = wl.decode_matrices(dv.small_model(layers=2, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.Q4, "bf16", wl.Q4)[m.layer] for m in mats]
    return dv.SweepInputs(mats, fmts, tokens=13)


@pytest.mark.parametrize("batch", [2, 4, 8, 16])
def test_batched_sweep_with_q4_equals_sequential(model_mixed, batch):
    """q4 and bf16 matrices in one table; batch 16 runs as passes of 8."""
    seq = run(model_mixed, 13, None)
    bat = run(model_mixed, 13, batch)
    for a, b in zip(seq, bat):
        assert np.array_equal(f32_bits(a), f32_bits(b))
