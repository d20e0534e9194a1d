"""A decode pass ordered against a framework stream (execution contract C3; Sec. 4.3): every
mechanism gives the plain sweep's outputs bit for bit, sees activations the framework stream writes
just before it (behind milliseconds of other work), and is seen by the framework's next operation."""
import numpy as np
import pytest
import torch

import oracle
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]
MODES = [wsr.WSR_ORDER_STREAM, wsr.WSR_ORDER_EVENT, wsr.WSR_ORDER_HOST_EVENT, wsr.WSR_ORDER_DRAIN]


@pytest.fixture(scope="module")
def model():
    mats = wl.decode_matrices(dv.small_model(layers=2, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.I8, wl.BF16, wl.Q4)[m.layer] for m in mats]
    return dv.SweepInputs(mats, fmts, tokens=1)


@pytest.fixture(scope="module")
def want_oracle(model):
    """The oracle's outputs of the pass, one vector per matrix."""
    ora, out = oracle.get(), []
    for i, fmt in enumerate(model.fmts):
        hw, x = model.host_weights(i), model.host_x(i, 0)
        out.append(ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x, threads=8) if fmt in (wl.Q4, wl.I8)
                   else ora.gemv16(hw, x, fmt, threads=8))
    return out


def plain(inp):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(inp.specs())
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    wsr.wsr_decode_sweep(mats, 1, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return [y.clone() for y in inp.y]


@pytest.mark.parametrize("mode", MODES, ids=lambda m: wsr.ORDER_NAMES[m].replace(" ", "_"))
def test_ordered_pass_sees_and_is_seen(model, want_oracle, mode):
    want = plain(model)
    xs = list(model.x.values())
    saved = [x[0].clone() for x, _ in xs]
    mats = wsr.make_mats(model.specs())
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    fs, own = torch.cuda.Stream(), torch.cuda.Stream()
    a = torch.randn(4096, 4096, device="cuda")
    torch.cuda.synchronize()
    for x, _ in xs:                       # activations the framework has not written yet
        x[0].fill_(0)
    for y in model.y:
        y.fill_(float("nan"))
    torch.cuda.synchronize()
    with torch.cuda.stream(fs):
        b = a
        for _ in range(6):                # milliseconds of framework work in flight
            b = torch.mm(b, a) * 1e-3
        for (x, _), s in zip(xs, saved):  # ... then it writes the pass's activations
            x[0].copy_(s)
    wsr.wsr_decode_sweep_ordered(mats, 1, ws, ws.numel(), fs, own, mode)
    with torch.cuda.stream(fs):           # the framework's next operation reads the outputs
        seen = [y.clone() for y in model.y]
    torch.cuda.synchronize()
    for i, (w, y, c) in enumerate(zip(want, model.y, seen)):
        got = y.cpu().numpy()
        assert rel_l2(got[0], want_oracle[i]) <= TOL, (wsr.ORDER_NAMES[mode], i)
        assert np.array_equal(f32_bits(w.cpu().numpy()), f32_bits(got)), (wsr.ORDER_NAMES[mode], i)
        assert np.array_equal(f32_bits(w.cpu().numpy()), f32_bits(c.cpu().numpy())), (wsr.ORDER_NAMES[mode], i)
    del b
