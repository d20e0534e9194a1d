"""Every GEMV entry point writes exactly rows [0, M) of each output column: a guard region after the
outputs (and between columns) keeps its sentinel for every row count modulo the row-group sizes."""
import numpy as np
import pytest
import torch

import synth
from synth import device as dv
from synth import workloads as wl
from gpu_util import needs_gpu, stream

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]
GUARD = 64
SENT = -12345.0


def guarded(M, T=1):
    y = torch.full((T, M + GUARD), SENT, dtype=torch.float32, device="cuda")
    return y


def check(y, M):
    y = y.cpu().numpy()
    assert (y[:, M:] == SENT).all(), np.nonzero(y[:, M:] != SENT)
    assert (y[:, :M] != SENT).all()


MS = [1, 2, 3, 5, 7, 8, 9, 13, 31, 33, 541, 995, 1001]


@pytest.mark.parametrize("M", MS)
def test_gemv_i8_rows_only(M):
    K = 512
    Wq = dv.to_device(synth.i8_codes(M, K, seed=1, stream=501))
    S = dv.to_device(synth.i8_scales(M, seed=1, stream=502))
    X = dv.to_device(synth.normal16((8, K), 1.0, "f16", seed=1, stream=503))
    y = guarded(M)
    wsr.wsr_gemv_i8(Wq, S, X[0], y, M, K, stream())
    check(y, M)
    for T in (1, 2, 4, 8):
        y = guarded(M, T)
        wsr.wsr_gemv_i8_cols(Wq, S, X, K * 2, y, (M + GUARD) * 4, M, K, T, stream())
        check(y, M)


@pytest.mark.parametrize("M", MS)
def test_gemv_q4_rows_only(M):
    for K in (512, 8192):
        Wq = dv.to_device(synth.q4_codes(M, K, seed=2, stream=511))
        S = dv.to_device(synth.q4_scales(M, K, seed=2, stream=512))
        X = dv.to_device(synth.normal16((8, K), 1.0, "f16", seed=2, stream=513))
        y = guarded(M)
        wsr.wsr_gemv_q4(Wq, S, X[0], y, M, K, stream())
        check(y, M)
        for T in (1, 2, 4, 8):
            y = guarded(M, T)
            wsr.wsr_gemv_q4_cols(Wq, S, X, K * 2, y, (M + GUARD) * 4, M, K, T, stream())
            check(y, M)


@pytest.mark.parametrize("M", MS)
def test_gemv16_rows_only(M):
    K = 512
    W = dv.to_device(synth.normal16((M, K), 0.02, "bf16", seed=3, stream=521))
    X = dv.to_device(synth.normal16((16, K), 1.0, "bf16", seed=3, stream=522))
    y = guarded(M)
    wsr.wsr_gemv_f16(W, X[0], y, M, K, wsr.WSR_BF16, stream())
    check(y, M)
    for T in (1, 2, 4, 8, 16):
        y = guarded(M, T)
        wsr.wsr_gemv_f16_cols(W, X, K * 2, y, (M + GUARD) * 4, M, K, T, wsr.WSR_BF16, stream())
        check(y, M)
