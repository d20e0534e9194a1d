"""Matrices whose byte size passes 4 GiB (64-bit offsets everywhere): one bf16, one q4 and one int8
matrix, each through its standalone GEMV and through the decode sweep, checked against the oracle
on sampled rows that include rows beyond the 4 GiB mark."""
import numpy as np
import pytest
import torch

import oracle
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]
K = 8192
CASES = {"bf16": (270_000, wl.BF16), "q4": (1_100_000, wl.Q4), "i8": (540_000, wl.I8)}


@pytest.mark.parametrize("name", list(CASES))
def test_matrix_over_4gib(name):
    M, fmt = CASES[name]
    mats = [wl.Mat(0, "big", 0, M, K, "attn")]
    inp = dv.SweepInputs(mats, [fmt], tokens=1)
    plane_row = {wl.BF16: 2 * K, wl.Q4: K // 2, wl.I8: K}[fmt]          # bytes per row of the weight plane
    assert M * plane_row > (4 << 30)
    spec = inp.specs()[0]
    y = inp.y[0][0]
    # standalone GEMV
    y.fill_(float("nan"))
    if fmt == wl.BF16:
        wsr.wsr_gemv_f16(spec["w"], spec["x"], y, M, K, wsr.WSR_BF16, stream())
    elif fmt == wl.Q4:
        wsr.wsr_gemv_q4(spec["w"], spec["scales"], spec["x"], y, M, K, stream())
    else:
        wsr.wsr_gemv_i8(spec["w"], spec["scales"], spec["x"], y, M, K, stream())
    torch.cuda.synchronize()
    gemv = y.cpu().numpy().copy()
    # decode sweep over the same matrix
    y.fill_(float("nan"))
    m = wsr.make_mats([spec])
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(m))
    wsr.wsr_decode_sweep(m, 1, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    swept = y.cpu().numpy()
    assert np.array_equal(f32_bits(gemv), f32_bits(swept))
    # sampled rows against the oracle: both ends, around the 4 GiB row, and spread rows
    edge = (4 << 30) // plane_row                                       # first row past 4 GiB
    rng = np.random.default_rng(M)
    rows = np.unique(np.concatenate([[0, 1, edge - 1, edge, edge + 1, M - 2, M - 1], rng.choice(M, 24, replace=False)]))
    ora = oracle.get()
    x = inp.host_x(0, 0)
    want = []
    for r in rows:
        hw = inp.host_weights(0, int(r), 1)
        want.append((ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt in (wl.Q4, wl.I8) else ora.gemv16(hw, x, fmt))[0])
    assert rel_l2(swept[rows], np.array(want)) <= TOL
    del inp, ws
    torch.cuda.empty_cache()
