"""The same kernels over host memory read in place across PCIe: results must be bitwise identical
to the HBM-resident runs (byte paths do not change outputs)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth import device as dv
from gpu_util import f32_bits, needs_gpu, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]


def pinned_copy(arr: np.ndarray) -> torch.Tensor:
    t = torch.empty(arr.nbytes, dtype=torch.uint8, pin_memory=True)
    t.numpy()[:] = np.ascontiguousarray(arr).view(np.uint8).ravel()
    return t


def test_register_pinned_host_and_probe():
    n = (1 << 22) + 5
    x = synth.grid_f32(n, seed=0, stream=301)
    page = 4096
    nbytes = (x.nbytes + page - 1) // page * page
    h = torch.zeros(nbytes, dtype=torch.uint8, pin_memory=True)
    h.numpy()[: x.nbytes] = x.view(np.uint8)
    assert h.data_ptr() % page == 0
    dev, granted = wsr.wsr_register_host(h, nbytes, 0)
    try:
        assert granted & wsr.WSR_REG_PREPINNED
        with pytest.raises(wsr.WsrError) as e:
            wsr.wsr_register_host(h, nbytes, 0)
        assert e.value.status == wsr.WSR_E_STATE
        out = torch.zeros(2, dtype=torch.float64, device="cuda")
        ws = zeros_u8(wsr.wsr_probe_workspace_bytes(n))
        wsr.wsr_probe_read(dev, n, out[0:], ws, ws.numel(), stream())
        wsr.wsr_probe_read(dv.to_device(x), n, out[1:], ws, ws.numel(), stream())
        torch.cuda.synchronize()
        mapped, resident = out.cpu().tolist()
        assert mapped == resident == oracle.get().probe_sum(x)
        # the mapped view aliases the host bytes: a host write is seen by the next read
        h.numpy()[:4] = np.frombuffer(np.float32(0.5).tobytes(), np.uint8)
        x2 = x.copy()
        x2[0] = 0.5
        wsr.wsr_probe_read(dev, n, out[0:], ws, ws.numel(), stream())
        torch.cuda.synchronize()
        assert out[0].item() == oracle.get().probe_sum(x2)
    finally:
        wsr.wsr_unregister_host(h)
    with pytest.raises(wsr.WsrError):
        wsr.wsr_unregister_host(h)


def test_unpinned_range_is_refused_without_pin_flag():
    page = 4096
    buf = np.zeros(4 * page + page, dtype=np.uint8)
    base = (buf.ctypes.data + page - 1) // page * page
    with pytest.raises(wsr.WsrError) as e:
        wsr.wsr_register_host(base, 4 * page, 0)
    assert e.value.status == wsr.WSR_E_UNSUPPORTED


@pytest.mark.parametrize("fmt", ["f16", "bf16", "q4"])
def test_gemv_host_mapped_bitwise(fmt):
    M, K = 2048, 4096
    x = synth.normal16(K, 1.0, "f16" if fmt == "q4" else fmt, seed=0, stream=302)
    dx = dv.to_device(x)
    yr = torch.empty(M, dtype=torch.float32, device="cuda")
    ym = torch.empty(M, dtype=torch.float32, device="cuda")
    if fmt == "q4":
        Wq = synth.q4_codes(M, K, seed=0, stream=303)
        S = synth.q4_scales(M, K, seed=0, stream=304)
        hq, hs = pinned_copy(Wq), pinned_copy(S)
        dq, gq = wsr.wsr_register_host(hq, hq.numel(), 0)
        ds, gs = wsr.wsr_register_host(hs, hs.numel(), 0)
        try:
            wsr.wsr_gemv_q4(dq, ds, dx, ym, M, K, stream())
            wsr.wsr_gemv_q4(dv.to_device(Wq), dv.to_device(S), dx, yr, M, K, stream())
            torch.cuda.synchronize()
        finally:
            wsr.wsr_unregister_host(hq)
            wsr.wsr_unregister_host(hs)
    else:
        W = synth.normal16((M, K), 0.02, fmt, seed=0, stream=305)
        hw = pinned_copy(W)
        dw, g = wsr.wsr_register_host(hw, hw.numel(), 0)
        try:
            f = wsr.WSR_F16 if fmt == "f16" else wsr.WSR_BF16
            wsr.wsr_gemv_f16(dw, dx, ym, M, K, f, stream())
            wsr.wsr_gemv_f16(dv.to_device(W), dx, yr, M, K, f, stream())
            torch.cuda.synchronize()
        finally:
            wsr.wsr_unregister_host(hw)
    assert np.array_equal(f32_bits(ym.cpu().numpy()), f32_bits(yr.cpu().numpy()))
