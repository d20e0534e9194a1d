"""The same kernels over host memory read in place across PCIe (the discrete-GPU case, Sec. 7.3):
results must equal the oracle within the stated tolerance and the HBM-resident runs bit for bit,
since byte paths do not change outputs (Sec. 5.2 and 6.2)."""
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


def _hip_runtime():
    """The HIP runtime this process already runs (the one PyTorch loaded), for exact-size pinned
    allocations that no caching allocator rounds or reuses."""
    import ctypes
    with open("/proc/self/maps") as f:
        path = next(l.split()[-1] for l in f if "libamdhip64" in l)
    hip = ctypes.CDLL(path)
    hip.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t, ctypes.c_uint]
    hip.hipHostFree.argtypes = [ctypes.c_void_p]
    return hip


def test_register_past_pinned_end_is_refused():
    """A range that starts inside a pinned allocation but runs past its end is refused before any
    kernel could read the unpinned pages; ranges inside the allocation are adopted.  No kernel is
    launched."""
    import ctypes
    page = 4096
    n = 1 << 20
    hip = _hip_runtime()
    torch.cuda.init()
    p = ctypes.c_void_p()
    assert hip.hipHostMalloc(ctypes.byref(p), n, 0) == 0
    base = p.value
    try:
        assert base % page == 0
        for off, nbytes in ((0, n + page), (0, n + (64 << 20)), (n - page, 2 * page)):
            with pytest.raises(wsr.WsrError) as e:
                wsr.wsr_register_host(base + off, nbytes, 0)
            assert e.value.status == wsr.WSR_E_SIZE, (off, nbytes, str(e.value))
        for off, nbytes in ((0, n), (page, 2 * page), (n - page, page)):
            dev, granted = wsr.wsr_register_host(base + off, nbytes, 0)
            try:
                assert granted & wsr.WSR_REG_PREPINNED and dev
            finally:
                wsr.wsr_unregister_host(base + off)
    finally:
        assert hip.hipHostFree(base) == 0


@pytest.mark.parametrize("fmt", ["f16", "bf16", "q4", "i8"])
def test_gemv_host_mapped_bitwise(fmt):
    """Each GEMV with its weights (and scales) in pinned host memory: within the tolerance of the
    oracle, and bit for bit the resident result."""
    M, K = 2048, 4096
    x = synth.normal16(K, 1.0, "f16" if fmt in ("q4", "i8") else fmt, seed=0, stream=302)
    dx = dv.to_device(x)
    yr = torch.empty(M, dtype=torch.float32, device="cuda")
    ym = torch.empty(M, dtype=torch.float32, device="cuda")
    ora = oracle.get()
    if fmt in ("q4", "i8"):
        if fmt == "q4":
            Wq = synth.q4_codes(M, K, seed=0, stream=303)
            S = synth.q4_scales(M, K, seed=0, stream=304)
            gemv, want = wsr.wsr_gemv_q4, ora.gemv_q4(Wq, S, x, threads=8)
        else:
            Wq = synth.i8_codes(M, K, seed=0, stream=303)
            S = synth.i8_scales(M, seed=0, stream=304)
            gemv, want = wsr.wsr_gemv_i8, ora.gemv_i8(Wq, S, x, threads=8)
        hq, hs = pinned_copy(Wq), pinned_copy(S)
        dq, gq = wsr.wsr_register_host(hq, hq.numel(), 0)
        ds, gs = wsr.wsr_register_host(hs, hs.numel(), 0)
        try:
            gemv(dq, ds, dx, ym, M, K, stream())
            gemv(dv.to_device(Wq), dv.to_device(S), dx, yr, M, K, stream())
            torch.cuda.synchronize()
        finally:
            wsr.wsr_unregister_host(hq)
            wsr.wsr_unregister_host(hs)
    else:
        W = synth.normal16((M, K), 0.02, fmt, seed=0, stream=305)
        want = ora.gemv16(W, x, fmt, threads=8)
        hw = pinned_copy(W)
        dw, g = wsr.wsr_register_host(hw, hw.numel(), 0)
        try:
            f = wsr.WSR_F16 if fmt == "f16" else wsr.WSR_BF16
            wsr.wsr_gemv_f16(dw, dx, ym, M, K, f, stream())
            wsr.wsr_gemv_f16(dv.to_device(W), dx, yr, M, K, f, stream())
            torch.cuda.synchronize()
        finally:
            wsr.wsr_unregister_host(hw)
    got = ym.cpu().numpy()
    assert rel_l2(got, want) <= TOL
    assert np.array_equal(f32_bits(got), f32_bits(yr.cpu().numpy()))


class MappedWeights:
    """Every weight and scale tensor of a resident SweepInputs copied into one pinned host buffer
    (each at a page boundary) and registered once; specs() gives the same table with the weight
    and scale pointers moved to the registered host view."""

    def __init__(self, inp):
        page = 4096
        tensors = [t for i in range(len(inp.mats)) for t in (inp.w[i], inp.s[i]) if t is not None]
        offs, total = {}, 0
        for t in tensors:
            offs[t.data_ptr()] = total
            total += -(-t.numel() * t.element_size() // page) * page
        self.host = torch.empty(total, dtype=torch.uint8, pin_memory=True)
        for t in tensors:
            o = offs[t.data_ptr()]
            nb = t.numel() * t.element_size()
            self.host[o:o + nb].copy_(t.reshape(-1).view(torch.uint8).cpu())
        self.dev, granted = wsr.wsr_register_host(self.host, total, 0)
        assert granted & wsr.WSR_REG_PREPINNED
        self.offs, self.inp = offs, inp

    def specs(self):
        out = self.inp.specs()
        for sp in out:
            sp["w"] = self.dev + self.offs[sp["w"].data_ptr()]
            if sp["scales"] is not None:
                sp["scales"] = self.dev + self.offs[sp["scales"].data_ptr()]
        return out

    def close(self):
        wsr.wsr_unregister_host(self.host)


@pytest.fixture(scope="module")
def mapped_model():
    """A mixed bf16 / q4 / int8 model and one int8 matrix at the protocol shape (12288 x 7168)."""
    mats = wl.decode_matrices(dv.small_model(layers=3, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.BF16, wl.Q4, wl.I8, wl.F16)[m.layer] for m in mats]
    mats.append(wl.Mat(len(mats), "protocol", 100, wl.PROTOCOL_M, wl.PROTOCOL_K, "attn"))
    fmts.append(wl.I8)
    inp = dv.SweepInputs(mats, fmts, tokens=3)
    mw = MappedWeights(inp)
    yield inp, mw
    mw.close()


def _sweep(inp, specs, tokens, batch=None):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(specs)
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    if batch is None:
        wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())
    else:
        wsr.wsr_decode_sweep_batched(mats, tokens, batch, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


def _oracle_rows(inp, i, t, rows):
    ora, fmt = oracle.get(), inp.fmts[i]
    x = inp.host_x(i, t)
    if rows is None:
        hw = inp.host_weights(i)
        return ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x, threads=8) if fmt in (wl.Q4, wl.I8) \
            else ora.gemv16(hw, x, fmt, threads=8)
    out = []
    for r in rows:
        hw = inp.host_weights(i, int(r), 1)
        out.append((ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x) if fmt in (wl.Q4, wl.I8)
                    else ora.gemv16(hw, x, fmt))[0])
    return np.array(out)


@pytest.mark.parametrize("batch", [None, 2, 4], ids=["sweep", "batched2", "batched4"])
def test_sweep_host_mapped(mapped_model, batch):
    """wsr_decode_sweep / wsr_decode_sweep_batched with every weight and scale read in place from
    registered host memory: every output of the small model against the oracle (all tokens), the
    protocol matrix on sampled rows, and all outputs bit for bit equal to the resident sweep."""
    inp, mw = mapped_model
    tokens = 3
    mapped = _sweep(inp, mw.specs(), tokens, batch)
    resident = _sweep(inp, inp.specs(), tokens, batch)
    for i, m in enumerate(inp.mats):
        assert np.array_equal(f32_bits(mapped[i]), f32_bits(resident[i])), (m.name, m.layer)
        big = m.M * m.K > (1 << 24)
        rows = np.unique(np.concatenate([[0, 1, m.M - 2, m.M - 1], np.linspace(0, m.M - 1, 12).astype(np.int64)])) \
            if big else None
        for t in ((0, tokens - 1) if big else range(tokens)):
            got = mapped[i][t] if rows is None else mapped[i][t][rows]
            assert rel_l2(got, _oracle_rows(inp, i, t, rows)) <= TOL, (m.name, m.layer, t)
