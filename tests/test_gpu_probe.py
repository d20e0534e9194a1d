"""Streaming-read probe on the GPU against the oracle: grid values sum exactly in double in any
order, so the GPU result must equal the oracle bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import device as dv
from synth import workloads as wl
from gpu_util import needs_gpu, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]


def probe(dbuf, n, ws=None):
    out = torch.zeros(1, dtype=torch.float64, device="cuda")
    if ws is None:
        ws = zeros_u8(wsr.wsr_probe_workspace_bytes(n))
    wsr.wsr_probe_read(dbuf if n else 0, n, out, ws, ws.numel(), stream())
    return out.item()


@pytest.mark.parametrize("n", [0, 1, 3, 4, 5, 1000, 8192, 8195, 256 * 8 * 4 * 2048 + 7, (1 << 22) + 1])
def test_probe_exact(n):
    x = synth.grid_f32(n, seed=0, stream=21)
    d = dv.to_device(x) if n else None
    assert probe(d, n) == oracle.get().probe_sum(x)


def test_probe_full_size_and_workspace_reuse():
    n = wl.PROBE_N
    x = synth.grid_f32(n, seed=0, stream=1)
    d = dv.to_device(x)
    ws = zeros_u8(wsr.wsr_probe_workspace_bytes(n))
    want = oracle.get().probe_sum(x)
    assert probe(d, n, ws) == want
    assert probe(d, n, ws) == want          # the workspace is left ready for the next call
    small = synth.grid_f32(777, seed=0, stream=2)
    assert probe(dv.to_device(small), 777, ws) == oracle.get().probe_sum(small)


def test_probe_closed_forms():
    n = 1_000_003
    assert probe(torch.full((n,), 0.375, device="cuda"), n) == n * 0.375
    half = synth.grid_f32(50_000, seed=0, stream=3)
    x = np.concatenate([half, -half[::-1]])
    assert probe(dv.to_device(x), x.size) == 0.0


def test_probe_general_values_within_rounding():
    rng = np.random.default_rng(5)
    n = 3_000_001
    x = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    got = probe(dv.to_device(x), n)
    want = oracle.get().probe_sum(x)
    assert abs(got - want) <= 2 * n * 2.0 ** -53 * float(np.abs(x.astype(np.float64)).sum())
    assert probe(dv.to_device(x), n) == got  # deterministic
