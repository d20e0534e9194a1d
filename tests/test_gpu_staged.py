"""Per-use copy endpoint (Sec. 8.1; Table 2's pipelined double-buffered copy): the staged sweep
copies each matrix through two device staging halves and must give the resident sweep's outputs bit
for bit, from pinned host, pageable host or device sources, with chunks that split matrices at
ragged row counts, and across back-to-back calls that reuse the staging buffer."""
import numpy as np
import pytest
import torch

import oracle
from synth import device as dv
from synth import workloads as wl
from gpu_util import TOL, f32_bits, needs_gpu, rel_l2, stream, zeros_u8

from paper_2608_12114_amd import wsr

pytestmark = [pytest.mark.gpu, needs_gpu]


@pytest.fixture(scope="module")
def model():
    mats = wl.decode_matrices(dv.small_model(layers=4, d=512, ffn=1536, vocab=3000))
    fmts = [(wl.I8, wl.Q4, wl.BF16, wl.F16, wl.I8)[m.layer] for m in mats]
    return dv.SweepInputs(mats, fmts, tokens=3)


def resident(inp, tokens):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(inp.specs())
    ws = zeros_u8(wsr.wsr_sweep_workspace_bytes(mats))
    wsr.wsr_decode_sweep(mats, tokens, ws, ws.numel(), stream())
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


def host_sources(inp, pinned):
    """Weights (and scales) of every matrix in host memory, regenerated from the seeds."""
    out = []
    for i in range(len(inp.mats)):
        hw = inp.host_weights(i)
        parts = hw if isinstance(hw, tuple) else (hw, None)
        keep = []
        for a in parts:
            if a is None:
                keep.append(None)
                continue
            a = np.ascontiguousarray(a)
            if pinned:
                t = torch.empty(a.nbytes, dtype=torch.uint8, pin_memory=True)
                t.numpy()[:] = a.view(np.uint8).ravel()
                keep.append(t)
            else:
                keep.append(a)
        out.append(keep)
    return out


def staged_specs(inp, sources):
    """Sweep specs whose weights and scales point at `sources`, which the caller keeps alive."""
    specs = inp.specs()
    for s, (w, sc) in zip(specs, sources):
        s["w"] = w.ctypes.data if isinstance(w, np.ndarray) else w
        s["scales"] = (sc.ctypes.data if isinstance(sc, np.ndarray) else sc) if sc is not None else None
    return specs


def run_staged(inp, specs, tokens, stage_bytes, same_stream=False, sync_each=True):
    for y in inp.y:
        y.fill_(float("nan"))
    mats = wsr.make_mats(specs)
    stage = zeros_u8(stage_bytes)
    cs = stream() if same_stream else torch.cuda.Stream()
    for t in range(tokens):
        wsr.wsr_sweep_staged(mats, t, stage, stage_bytes, stream(), cs)
        if sync_each:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    return [y.cpu().numpy().copy() for y in inp.y]


@pytest.mark.parametrize("source", ["pinned", "pageable", "device"])
@pytest.mark.parametrize("stage_kib", [64, 1000, 16384])
def test_staged_equals_resident(model, source, stage_kib):
    """64 KiB halves of 32 KiB split every matrix into chunks of a few rows (and at ragged counts);
    16 MiB holds whole matrices."""
    want = resident(model, 3)
    src = None if source == "device" else host_sources(model, source == "pinned")   # kept alive
    specs = model.specs() if src is None else staged_specs(model, src)
    got = run_staged(model, specs, 3, stage_kib << 10)
    for i, (a, b) in enumerate(zip(want, got)):
        assert np.array_equal(f32_bits(a), f32_bits(b)), (source, stage_kib, model.mats[i].name, model.mats[i].layer)


def test_staged_back_to_back_and_same_stream(model):
    """Tokens enqueued back to back reuse the staging buffer without host synchronisation; copies
    and GEMVs on one stream also work (serially); pinned and pageable sources."""
    want = resident(model, 3)
    for pinned in (True, False):
        src = host_sources(model, pinned)
        specs = staged_specs(model, src)
        for same in (False, True):
            for kib in (96, 1000):
                got = run_staged(model, specs, 3, kib << 10, same_stream=same, sync_each=False)
                for a, b in zip(want, got):
                    assert np.array_equal(f32_bits(a), f32_bits(b)), (pinned, same, kib)


def test_staged_parity_with_oracle(model):
    src = host_sources(model, True)
    specs = staged_specs(model, src)
    got = run_staged(model, specs, 2, 256 << 10)
    ora = oracle.get()
    for i, fmt in enumerate(model.fmts):
        x = model.host_x(i, 1)
        hw = model.host_weights(i)
        want = ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x, 8) if fmt in (wl.Q4, wl.I8) else ora.gemv16(hw, x, fmt, threads=8)
        assert rel_l2(got[i][1], want) <= TOL, (i, fmt)


def test_staged_protocol_size():
    """Two of the protocol's 12288 x 7168 int8 matrices from pinned host memory through 2 x 32 MiB
    of staging, against the resident sweep."""
    mats = wl.protocol_matrices(n=2)
    inp = dv.SweepInputs(mats, [wl.I8] * 2, tokens=1)
    want = resident(inp, 1)
    src = host_sources(inp, True)
    specs = staged_specs(inp, src)
    got = run_staged(inp, specs, 1, 64 << 20)
    for a, b in zip(want, got):
        assert np.array_equal(f32_bits(a), f32_bits(b))


def test_staged_from_several_threads(model):
    """Four host threads run staged sweeps at once, each with its own streams, staging buffer and
    outputs, from the same pinned sources: the per-device events are created once and every call's
    enqueueing is serialised, so each thread gets the resident outputs bit for bit."""
    import threading
    want = resident(model, 3)
    src = host_sources(model, True)
    base = staged_specs(model, src)
    outs, errs = [], []
    jobs = []
    for _ in range(4):
        ys = [torch.full_like(y, float("nan")) for y in model.y]
        specs = [dict(s, y=y) for s, y in zip(base, ys)]
        jobs.append((wsr.make_mats(specs), ys, zeros_u8(96 << 10), torch.cuda.Stream(), torch.cuda.Stream()))
    torch.cuda.synchronize()

    def work(mats, stage, s, cs):
        try:
            for t in range(3):
                wsr.wsr_sweep_staged(mats, t, stage, stage.numel(), s, cs)
        except Exception as e:          # reported below, on the test's thread
            errs.append(e)

    threads = [threading.Thread(target=work, args=(m, st, s, cs)) for m, _, st, s, cs in jobs]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errs, errs
    for k, (_, ys, *_rest) in enumerate(jobs):
        for i, (a, y) in enumerate(zip(want, ys)):
            assert np.array_equal(f32_bits(a), f32_bits(y.cpu().numpy())), (k, i)
