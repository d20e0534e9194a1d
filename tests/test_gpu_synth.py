"""The GPU copy of the input generator draws exactly the host generator's values."""
import numpy as np
import pytest
import torch

import synth
from synth import device as dv
from gpu_util import needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]


@pytest.mark.parametrize("fmt,sigma", [("f16", 0.02), ("bf16", 0.02), ("f16", 1.0), ("bf16", 1.0)])
@pytest.mark.parametrize("n,e0", [(1, 0), (7, 3), (100_003, 0), (4_000_001, 12_345)])
def test_normal16_device_equals_host(fmt, sigma, n, e0):
    t = torch.empty(n, dtype=torch.int16, device="cuda")
    dv.gen_normal16(t, sigma, fmt, seed=5, stream=77, e0=e0)
    host = synth.normal16(n, sigma, fmt, seed=5, stream=77, e0=e0)
    assert np.array_equal(t.cpu().numpy().view(np.uint16), host)


@pytest.mark.parametrize("nbytes,row0", [(1, 0), (9, 0), (1_000_001, 3)])
def test_q4_scales_grid_device_equal_host(nbytes, row0):
    K = 64
    t = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dv.gen_q4(t, seed=1, stream=9, e0=row0 * K)
    host = np.empty(nbytes, np.uint8)
    synth.lib().synth_q4(host.ctypes.data, nbytes, 1, 9, row0 * K, 4)
    assert np.array_equal(t.cpu().numpy(), host)
    s = torch.empty(nbytes, dtype=torch.int16, device="cuda")
    dv.gen_uniform16(s, 0.005, 0.02, "f16", seed=1, stream=10, e0=row0)
    assert np.array_equal(s.cpu().numpy().view(np.uint16),
                          synth.uniform16(nbytes, 0.005, 0.02, "f16", seed=1, stream=10, e0=row0))
    g = torch.empty(nbytes, dtype=torch.float32, device="cuda")
    dv.gen_grid_f32(g, seed=1, stream=11, e0=row0)
    assert np.array_equal(g.cpu().numpy(), synth.grid_f32(nbytes, seed=1, stream=11, e0=row0))


@pytest.mark.parametrize("n,e0", [(1, 0), (4099, 7), (1 << 20, 123456789)])
def test_i8_device_equals_host(n, e0):
    t = torch.empty(n, dtype=torch.int8, device="cuda")
    dv.gen_i8(t, seed=2, stream=13, e0=e0)
    host = np.empty(n, np.int8)
    synth.lib().synth_i8(host.ctypes.data, n, 2, 13, e0, 4)
    assert np.array_equal(t.cpu().numpy(), host)
