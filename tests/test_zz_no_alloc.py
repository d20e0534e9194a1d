"""wsr_decode_sweep_noalloc, the sweep for callers that cannot allocate device memory: its outputs
equal wsr_decode_sweep's bit for bit (same kernels, the library's scratch in place of the caller's
workspace) on consecutive calls that share that scratch, the second with a smaller table, and they
match the oracle."""
import numpy as np
import pytest
import torch

import oracle
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]


def _run(inp, tokens, call, chained=False):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(inp.specs(chained=chained))
    call(mats, tokens)
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


def _with_ws(mats, tokens):
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())


def _noalloc(mats, tokens):
    wsr.wsr_decode_sweep_noalloc(mats, tokens, stream())


def _check(inp, tokens, chained=False):
    want = _run(inp, tokens, _with_ws, chained)
    got = _run(inp, tokens, _noalloc, chained)
    ora = oracle.get()
    for i, (m, fmt) in enumerate(zip(inp.mats, inp.fmts)):
        assert np.array_equal(f32_bits(got[i]), f32_bits(want[i])), (m.name, m.layer)
        hw = inp.host_weights(i)
        for t in (0, tokens - 1):
            x = inp.host_x(i, t)
            yo = ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt in (wl.Q4, wl.I8) else ora.gemv16(hw, x, fmt)
            assert rel_l2(got[i][t], yo) <= TOL, (m.name, m.layer, t)


def test_noalloc_two_calls_second_smaller():
    """A mixed-format model (one launch per token), then a smaller bf16 model (claimed tiles, whose
    counters live in the scratch) in the next call, then the first model again with dependency
    boundaries (several launches per token)."""
    big = wl.decode_matrices(dv.small_model(layers=3, d=512, ffn=1536, vocab=3000))
    big_in = dv.SweepInputs(big, [(wl.Q4, wl.BF16, wl.I8, wl.F16)[m.layer] for m in big], tokens=3)
    small = wl.decode_matrices(dv.small_model(layers=1, d=256, ffn=512, vocab=700))
    small_in = dv.SweepInputs(small, [wl.BF16] * len(small), tokens=2)
    assert len(small) < len(big)
    _check(big_in, 3)
    _check(small_in, 2)
    _check(big_in, 3, chained=True)


def test_noalloc_table_too_large_is_refused():
    good = dict(fmt=wsr.WSR_BF16, M=8, K=64, w=0x10000, x=0x10000, y=0x10000, x_tok_stride=128, y_tok_stride=32)
    mats = wsr.make_mats([good] * 6000)
    with pytest.raises(wsr.WsrError) as e:
        wsr.wsr_decode_sweep_noalloc(mats, 1, stream())
    assert e.value.status == wsr.WSR_E_SIZE
